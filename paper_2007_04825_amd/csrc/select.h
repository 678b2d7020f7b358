// Wave-level top-k selection for the improved-clustered attention (Section 3.3).
#pragma once
#include "common.h"

namespace ca {

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
template <typename KeyFn, typename OutT>
__device__ int wave_select_topk(KeyFn key, int m, int kk, int* hist, OutT* out) {
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
    bin = __builtin_amdgcn_readlane(bin, leader);
    above = __builtin_amdgcn_readlane(above, leader);
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
    if (sel) out[written + __popcll(selmask & lanemask_lt())] = static_cast<OutT>(pos);
    written += __popcll(selmask);
    eq_seen += __popcll(eqmask);
  }
  return written;
}

// The kk-th largest of the keys held by the wave (k1 in every lane, plus k2
// when two is set; key 0 stands for "no value"): the largest T with at least
// kk keys >= T, built one bit at a time from the most significant down with
// wave ballots (no LDS traffic).  Requires kk <= number of nonzero keys.
__device__ __forceinline__ uint32_t wave_kth_key(uint32_t k1, uint32_t k2, bool two, int kk) {
  uint32_t t = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t cand = t | (1u << bit);
    int cnt = __popcll(__ballot(k1 >= cand));
    if (two) cnt += __popcll(__ballot(k2 >= cand));
    if (cnt >= kk) t = cand;
  }
  return t;
}

// Top-kk (1 <= kk <= 128, kk <= m) of row[0..m) by value, ties to the smaller
// position, for one wave.  row may live in LDS or global memory.  Writes the
// chosen positions in ascending order to out[] and returns their number (kk);
// also returns the row maximum and z = sum_pos exp(row[pos] - max).
//
// Each lane keeps the largest and the second largest value of its strided
// slice.  The kk-th largest of those values is a threshold tau
// that at least kk entries reach, so every entry of the top-kk set is >= tau.
// One more sweep collects the entries >= tau in position order (usually
// little more than kk of them); the exact kk-th value among them is found by
// the same bitwise search, and the entries above it plus the first ones equal
// to it (smallest positions) are kept.  If more than CAP entries reach tau
// (many ties) the radix selection above runs instead.
// scratch: 2*CAP ints of LDS private to the wave (candidate values, then
// candidate positions; the whole area is the radix histogram of the fallback).
template <int CAP, typename OutT>
__device__ int wave_topk_row(const float* row, int m, int kk, int* scratch, OutT* out,
                             float* mx_out, float* z_out) {
  static_assert(2 * CAP >= 256 && CAP <= 128, "scratch layout");
  float* cval = reinterpret_cast<float*>(scratch);
  int* cpos = scratch + CAP;
  const int lane = lane_id();
  float a1 = -INFINITY, a2 = -INFINITY;
  int have = 0;
  // eight loads in flight per lane (the row may be in global memory)
#pragma unroll 8
  for (int pos = lane; pos < m; pos += 64) {
    const float x = row[pos];
    a2 = fmaxf(a2, fminf(a1, x));
    a1 = fmaxf(a1, x);
    ++have;
  }
  const float mx = wave_max(a1);
  // the threshold from both kept values of every lane whenever a lane saw two:
  // the kk-th largest of up to 128 values lets fewer entries through than the
  // kk-th of the 64 lane maxima (long rows fell back to the radix selection)
  const bool two = kk > 64 || m > 64;
  const uint32_t tau = wave_kth_key(have > 0 ? order_key(a1) : 0u, have > 1 ? order_key(a2) : 0u,
                                    two, kk);
  float z = 0.0f;
  int c = 0;
#pragma unroll 8
  for (int base = 0; base < m; base += 64) {
    const int pos = base + lane;
    const bool ok = pos < m;
    const float x = ok ? row[pos] : -INFINITY;
    z += ok ? __expf(x - mx) : 0.0f;
    const bool sel = ok && order_key(x) >= tau;
    const uint64_t bal = __ballot(sel);
    const int idx = c + __popcll(bal & lanemask_lt());
    if (sel && idx < CAP) {
      cval[idx] = x;
      cpos[idx] = pos;
    }
    c += __popcll(bal);
  }
  z = wave_sum(z);
  *mx_out = mx;
  *z_out = z;
  wave_lds_sync();
  if (c > CAP) {
    return wave_select_topk([&](int pos) { return order_key(row[pos]); }, m, kk, scratch, out);
  }
  const uint32_t kc1 = lane < c ? order_key(cval[lane]) : 0u;
  const uint32_t kc2 = lane + 64 < c ? order_key(cval[lane + 64]) : 0u;
  const uint32_t kth = wave_kth_key(kc1, kc2, c > 64, kk);
  const int need = kk - __popcll(__ballot(kc1 > kth)) - __popcll(__ballot(kc2 > kth));
  int written = 0, eq_seen = 0;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int i = lane + 64 * r;
    const uint32_t key = r ? kc2 : kc1;
    const bool valid = i < c;
    const bool eq = valid && key == kth;
    const uint64_t eqmask = __ballot(eq);
    const bool sel = (valid && key > kth) || (eq && eq_seen + __popcll(eqmask & lanemask_lt()) < need);
    const uint64_t selmask = __ballot(sel);
    if (sel) out[written + __popcll(selmask & lanemask_lt())] = static_cast<OutT>(cpos[i]);
    written += __popcll(selmask);
    eq_seen += __popcll(eqmask);
  }
  wave_lds_sync();
  return written;
}

// ---------------------------------------------------------------------------
// Rows handled by lane groups: with GL-lane groups (GL = 16 or 32), group
// g = lane / GL owns a row and lane c = lane % GL of the group reads positions
// c, c + GL, c + 2 GL, ...  Reductions stay inside a group: DPP row operations
// within 16 lanes and, for 32-lane groups, one swap between the two rows.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int row16_sum_i(int x) {
  x += dpp_i<0xB1>(x);
  x += dpp_i<0x4E>(x);
  x += dpp_i<0x141>(x);
  return x + dpp_i<0x140>(x);
}
__device__ __forceinline__ uint32_t row16_and(uint32_t x) {
  x &= static_cast<uint32_t>(dpp_i<0xB1>(static_cast<int>(x)));
  x &= static_cast<uint32_t>(dpp_i<0x4E>(static_cast<int>(x)));
  x &= static_cast<uint32_t>(dpp_i<0x141>(static_cast<int>(x)));
  return x & static_cast<uint32_t>(dpp_i<0x140>(static_cast<int>(x)));
}
__device__ __forceinline__ uint32_t row16_or(uint32_t x) {
  x |= static_cast<uint32_t>(dpp_i<0xB1>(static_cast<int>(x)));
  x |= static_cast<uint32_t>(dpp_i<0x4E>(static_cast<int>(x)));
  x |= static_cast<uint32_t>(dpp_i<0x141>(static_cast<int>(x)));
  return x | static_cast<uint32_t>(dpp_i<0x140>(static_cast<int>(x)));
}
__device__ __forceinline__ int wave_max_i(int x) {
  x = max(x, dpp_i<0xB1>(x));
  x = max(x, dpp_i<0x4E>(x));
  x = max(x, dpp_i<0x141>(x));
  x = max(x, dpp_i<0x140>(x));
  return cross_rows_max(x);
}

template <int GL> __device__ __forceinline__ int grp_sum_i(int x) {
  x = row16_sum_i(x);
  if constexpr (GL == 32) x += lane_xor16(x);
  return x;
}
template <int GL> __device__ __forceinline__ float grp_sum(float x) {
  x = row16_sum(x);
  if constexpr (GL == 32) x += lane_xor16(x);
  return x;
}
template <int GL> __device__ __forceinline__ float grp_max(float x) {
  x = row16_max(x);
  if constexpr (GL == 32) x = fmaxf(x, lane_xor16(x));
  return x;
}
template <int GL> __device__ __forceinline__ uint32_t grp_min_u(uint32_t x) {
  x = min(x, static_cast<uint32_t>(dpp_i<0xB1>(static_cast<int>(x))));
  x = min(x, static_cast<uint32_t>(dpp_i<0x4E>(static_cast<int>(x))));
  x = min(x, static_cast<uint32_t>(dpp_i<0x141>(static_cast<int>(x))));
  x = min(x, static_cast<uint32_t>(dpp_i<0x140>(static_cast<int>(x))));
  if constexpr (GL == 32) x = min(x, lane_xor16_u(x));
  return x;
}
template <int GL> __device__ __forceinline__ int grp_max_i(int x) {
  x = max(x, dpp_i<0xB1>(x));
  x = max(x, dpp_i<0x4E>(x));
  x = max(x, dpp_i<0x141>(x));
  x = max(x, dpp_i<0x140>(x));
  if constexpr (GL == 32) x = max(x, lane_xor16(x));
  return x;
}
template <int GL> __device__ __forceinline__ uint32_t grp_and(uint32_t x) {
  x = row16_and(x);
  if constexpr (GL == 32) x &= lane_xor16_u(x);
  return x;
}
template <int GL> __device__ __forceinline__ uint32_t grp_or(uint32_t x) {
  x = row16_or(x);
  if constexpr (GL == 32) x |= lane_xor16_u(x);
  return x;
}
// This lane's group's bits of a wave ballot, and the lanes of the group below this one.
template <int GL> __device__ __forceinline__ uint32_t grp_field(uint64_t ballot) {
  const uint64_t f = ballot >> (threadIdx.x & (64 - GL));
  return GL == 32 ? static_cast<uint32_t>(f) : static_cast<uint32_t>(f) & 0xffffu;
}
template <int GL> __device__ __forceinline__ uint32_t grp_lanemask_lt() {
  return (1u << (threadIdx.x & (GL - 1))) - 1u;
}
// Inclusive prefix sum over the lanes of this lane's group.
template <int GL> __device__ __forceinline__ int grp_incl_scan_i(int x) {
  x += dpp_i<0x111>(x);  // row_shr:1 (lanes shifted in from outside the row read 0)
  x += dpp_i<0x112>(x);  // row_shr:2
  x += dpp_i<0x114>(x);  // row_shr:4
  x += dpp_i<0x118>(x);  // row_shr:8
  if constexpr (GL == 32) {
    const int r15 = __builtin_amdgcn_readlane(x, 15), r47 = __builtin_amdgcn_readlane(x, 47);
    if (threadIdx.x & 16) x += (threadIdx.x & 32) ? r47 : r15;
  }
  return x;
}
// Positions per lane when a group sweeps a row of m <= 32 GL entries in
// contiguous blocks: ceil(m / GL), made odd where that stays within 32 so
// that the lanes' LDS reads fall in distinct banks.
template <int GL> __device__ __forceinline__ int grp_block_len(int m) {
  const int l = (m + GL - 1) / GL;
  return (l & 1) || l >= 32 ? l : l + 1;
}
// A float f with (x >= f) == (order_key(x) >= tau) for every finite x.
__device__ __forceinline__ float key_threshold(uint32_t tau) {
  if (tau > 0xff7fffffu) return INFINITY;  // above every finite key
  tau = tau > 0x00800000u ? tau : 0x00800000u;  // every finite key is at least this
  return __uint_as_float((tau & 0x80000000u) ? (tau & 0x7fffffffu) : ~tau);
}

// A threshold for the kk largest of the keys held by the group (NK per lane,
// 0 = none), built one bit at a time from the most significant down: the
// largest T with at least kk keys >= T (the kk-th largest key), unless a
// prefix that exactly kk keys reach turns up first, which ends the group's
// search (the same keys reach it: the kk largest).  The bits that all of the
// group's keys share are taken as they are, so the search starts at the
// highest bit where they differ; the loop runs to the wave's highest such bit
// or until every group has stopped, and the extra steps leave a group's
// result unchanged.  kk = 0 gives 0xffffffff (nothing reaches it).
template <int NK, int GL>
__device__ __forceinline__ uint32_t group_kth_key(const uint32_t* keys, int kk) {
  uint32_t a = 0xffffffffu, o = 0u;
#pragma unroll
  for (int e = 0; e < NK; ++e) {
    if (keys[e] != 0u) {
      a &= keys[e];
      o |= keys[e];
    }
  }
  a = grp_and<GL>(a);
  o = grp_or<GL>(o);
  const uint32_t diff = (o != 0u) ? (a ^ o) : 0u;
  const int hb = diff != 0u ? 31 - __clz(static_cast<int>(diff)) : -1;
  uint32_t t = hb >= 0 ? (o & ~((2u << hb) - 1u)) : o;  // the common prefix, zeros below
  const int top = __builtin_amdgcn_readfirstlane(wave_max_i(hb));  // uniform loop bound
  // a group stops as soon as exactly kk keys reach t: every later step would
  // keep that same set of keys
  bool done = kk <= 0;
  for (int bit = top; bit >= 0; --bit) {
    if (__ballot(!done) == 0ull) break;
    const uint32_t cand = t | (1u << bit);
    // the group's count from one ballot per key slot (no cross-lane chain)
    int tot = 0;
#pragma unroll
    for (int e = 0; e < NK; ++e) tot += __popc(grp_field<GL>(__ballot(keys[e] >= cand)));
    if (!done && tot >= kk) {
      t = cand;
      done = tot == kk;
    }
  }
  return kk > 0 ? t : 0xffffffffu;
}

// Top-kk positions of the group's row row[0..m) (0 <= kk, kk <= m), ties to
// the smaller position, given a threshold tau that every top-kk entry reaches
// (its order key).  The row is read up to GL * grp_block_len(m), and the
// entries from m on must be -inf: one sweep lists the positions with key >= tau in ascending
// order in cand[0..CAP); unless exactly kk reached tau in every row of the
// wave, the exact kk-th key among them is found by a second search, and the
// entries above it plus the first ones equal to it are compacted in place.
// Returns the number selected (kk), or -1 if more than CAP positions reached
// tau (the caller then selects that row another way).
template <int CAP, int GL>
__device__ int group_select(const float* row, int m, int kk, uint32_t tau, uint16_t* cand) {
  static_assert(CAP % GL == 0 && CAP <= 256, "candidate layout");
  constexpr int PER = CAP / GL;
  const int c = threadIdx.x & (GL - 1);
  const uint32_t lt = grp_lanemask_lt<GL>();
  // each lane sweeps its own block of L consecutive positions, so lane order
  // is position order, and one prefix sum over the group places every
  // lane's hits
  const int L = grp_block_len<GL>(m);
  const int base = c * L;
  const float tf = key_threshold(tau);
  uint32_t hits = 0u;  // bit i: position base + i reaches tau
  if (L == 32) {
    // a block of 32 (a full row of 32 GL entries) would put the group's reads
    // in one bank: each lane starts its sweep at offset c of its block and
    // wraps around, collecting the bits in that rotated order
#pragma unroll
    for (int i0 = 0; i0 < 32; i0 += 8) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = row[base + ((i0 + e + c) & 31)];
#pragma unroll
      for (int e = 0; e < 8; ++e) hits |= x[e] >= tf ? (1u << (i0 + e)) : 0u;
    }
    hits = __builtin_rotateleft32(hits, static_cast<uint32_t>(c));
  } else {
    // an odd block length puts the group's reads in distinct banks
    for (int i0 = 0; i0 < L; i0 += 8) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = i0 + e < L ? row[base + i0 + e] : -INFINITY;
      uint32_t h8 = 0u;
#pragma unroll
      for (int e = 0; e < 8; ++e) h8 |= x[e] >= tf ? (1u << e) : 0u;
      hits |= h8 << i0;
    }
  }
  const int mine = __popc(hits);
  const int cnt = grp_sum_i<GL>(mine);
  if (cnt > CAP) return -1;
  int at = grp_incl_scan_i<GL>(mine) - mine;
  while (hits != 0u) {
    const int i = __ffs(static_cast<int>(hits)) - 1;
    hits &= hits - 1u;
    cand[at++] = static_cast<uint16_t>(base + i);
  }
  wave_lds_sync();
  if (__ballot(cnt != kk) == 0ull) return cnt;
  int pos[PER];
  uint32_t ck[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int i = c + GL * e;
    pos[e] = i < cnt ? cand[i] : 0;
  }
#pragma unroll
  for (int e = 0; e < PER; ++e) ck[e] = c + GL * e < cnt ? order_key(row[pos[e]]) : 0u;
  // A few entries past the top kk (the usual case: the threshold misses only
  // the entries of slices that hold more top entries than they keep) are
  // dropped one at a time, each the last candidate in (key descending,
  // position ascending) order: the smallest key, the last position among
  // equal ones.  That leaves the same kk entries as the search below, in far
  // fewer steps.
  constexpr int kDropMax = 8;
  const int extra = cnt - kk;  // the same in every lane of the group
  if (__ballot(extra > kDropMax) == 0ull) {
    bool live[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) live[e] = c + GL * e < cnt;
    for (int it = 0; it < kDropMax; ++it) {
      if (__ballot(it < extra) == 0ull) break;
      uint32_t m = 0xffffffffu;
#pragma unroll
      for (int e = 0; e < PER; ++e) m = live[e] && ck[e] < m ? ck[e] : m;
      m = grp_min_u<GL>(m);
      int last = -1;
#pragma unroll
      for (int e = 0; e < PER; ++e) last = live[e] && ck[e] == m ? c + GL * e : last;
      last = grp_max_i<GL>(last);
      if (it < extra) {
#pragma unroll
        for (int e = 0; e < PER; ++e) live[e] = live[e] && c + GL * e != last;
      }
    }
    wave_lds_sync();
    int written = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const uint32_t sf = grp_field<GL>(__ballot(live[e]));
      if (live[e]) cand[written + __popc(sf & lt)] = static_cast<uint16_t>(pos[e]);
      written += __popc(sf);
    }
    wave_lds_sync();
    return written;
  }
  const uint32_t kth = group_kth_key<PER, GL>(ck, kk);
  int gt = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) gt += ck[e] > kth ? 1 : 0;
  const int need = kk - grp_sum_i<GL>(gt);
  wave_lds_sync();
  int written = 0, eq_seen = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const bool eq = ck[e] == kth;  // key 0 (no entry) never equals kth > 0
    const uint32_t ef = grp_field<GL>(__ballot(eq));
    const bool sel = ck[e] > kth || (eq && eq_seen + __popc(ef & lt) < need);
    const uint32_t sf = grp_field<GL>(__ballot(sel));
    if (sel) cand[written + __popc(sf & lt)] = static_cast<uint16_t>(pos[e]);
    written += __popc(sf);
    eq_seen += __popc(ef);
  }
  wave_lds_sync();
  return written;
}

// Threshold for group_select from the row itself: each lane keeps the NT
// largest values of its positions; the kk-th largest of those GL * NT values
// (GL * NT >= kk) is reached by every top-kk entry.
template <int NT, int GL>
__device__ uint32_t group_row_threshold(const float* row, int m, int kk) {
  constexpr int SW = 64 / GL;
  const int c = threadIdx.x & (GL - 1);
  float top[NT];
#pragma unroll
  for (int e = 0; e < NT; ++e) top[e] = -INFINITY;
  for (int i0 = 0; i0 < m; i0 += SW * GL) {
    float x[SW];
#pragma unroll
    for (int e = 0; e < SW; ++e) {
      const int p = i0 + GL * e + c;
      x[e] = p < m ? row[p] : -INFINITY;
    }
#pragma unroll
    for (int e = 0; e < SW; ++e) {
      float v = x[e];
#pragma unroll
      for (int t = 0; t < NT; ++t) {  // insertion into the descending list
        const float hi = fmaxf(top[t], v);
        v = fminf(top[t], v);
        top[t] = hi;
      }
    }
  }
  uint32_t keys[NT];
#pragma unroll
  for (int e = 0; e < NT; ++e) keys[e] = top[e] > -INFINITY ? order_key(top[e]) : 0u;
  return group_kth_key<NT, GL>(keys, kk);
}

}  // namespace ca
