// Wave-level top-k selection for the improved-clustered attention (Section 3.3).
#pragma once
#include "common.h"

namespace ca {

// Makes the LDS writes of this wave visible to its other lanes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Selects the kk positions of [0, m) with the largest keys, where
// key(pos) = order_key(value) for a valid position and 0 for an invalid one;
// among equal keys the smaller positions win.  Writes the chosen positions in
// ascending order to out[0..kk) and returns how many were written (kk, or the
// number of valid positions if that is smaller).
//
// Radix select on the 32-bit keys, one 8-bit digit per pass from the most
// significant down: a 256-bin histogram (hist, 256 ints of LDS private to the
// wave) of the candidates that match the digits fixed so far locates the
// digit of the kk-th key.  After four passes the kk-th key T is known, and a
// single ordered sweep takes every key > T and the first (kk - #(> T)) keys
// equal to T.
template <typename KeyFn>
__device__ int wave_select_topk(KeyFn key, int m, int kk, int* hist, int* out) {
  const int lane = lane_id();
  if (kk <= 0 || m <= 0) return 0;
  uint32_t prefix = 0, pmask = 0;
  int need = kk;
  bool all_valid = false;
  for (int shift = 24; shift >= 0; shift -= 8) {
#pragma unroll
    for (int e = 0; e < 4; ++e) hist[lane * 4 + e] = 0;
    wave_lds_sync();
    for (int pos = lane; pos < m; pos += 64) {
      const uint32_t kx = key(pos);
      if (kx != 0u && (kx & pmask) == prefix) atomicAdd(&hist[(kx >> shift) & 255u], 1);
    }
    wave_lds_sync();
    // lane l owns bins 255-4l, 254-4l, 253-4l, 252-4l (descending)
    int c[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) c[e] = hist[255 - (4 * lane + e)];
    const int local = c[0] + c[1] + c[2] + c[3];
    const int incl = wave_incl_scan(local);
    const int excl = incl - local;
    const uint64_t found = __ballot(excl < need && incl >= need);
    if (found == 0) {  // fewer valid keys than kk: take them all
      all_valid = true;
      break;
    }
    const int leader = __ffsll(static_cast<unsigned long long>(found)) - 1;
    int bin = 0, above = excl;
    if (lane == leader) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (above + c[e] >= need) {
          bin = 255 - (4 * lane + e);
          break;
        }
        above += c[e];
      }
    }
    bin = __shfl(bin, leader);
    above = __shfl(above, leader);
    prefix |= static_cast<uint32_t>(bin) << shift;
    pmask |= 0xffu << shift;
    need -= above;
    wave_lds_sync();
  }
  const uint32_t thr = all_valid ? 0u : prefix;
  if (all_valid) need = 0;
  int written = 0, eq_seen = 0;
  for (int base = 0; base < m; base += 64) {
    const int pos = base + lane;
    const uint32_t kx = pos < m ? key(pos) : 0u;
    const bool gt = kx > thr;
    const bool eq = !all_valid && kx == thr;
    const uint64_t eqmask = __ballot(eq);
    const int eq_rank = eq_seen + __popcll(eqmask & lanemask_lt());
    const bool sel = gt || (eq && eq_rank < need);
    const uint64_t selmask = __ballot(sel);
    if (sel) out[written + __popcll(selmask & lanemask_lt())] = pos;
    written += __popcll(selmask);
    eq_seen += __popcll(eqmask);
  }
  return written;
}

}  // namespace ca
