// K-means in Hamming space on the hash codes (Section 3.2.2), and the
// cluster-sorted member lists (CSR) that the later stages read.
//
// Assign step on the int8 matrix cores.  A code h is expanded to a 64-entry
// int8 vector: bit b (b < n_bits) becomes +64 / -64 for a query and +16 / -16
// for a centroid, positions n_bits..63 are 0.  One v_mfma_i32_16x16x64_i8
// over the 16 centroids j = 16 t + r of tile t, its accumulator starting at
// kTie - r, gives per query 1024 * (n_bits - 2 * ham) + kTie - r.  The tile's
// part -16 t comes from position 63 when n_bits <= 63 (query +16, centroid
// -t), and is otherwise taken off each tile's maximum, so that
//     key = 1024 * (n_bits - 2 * ham(h, c_j)) + kTie - j      (kTie = 1023)
// and the largest key is the nearest centroid with ties resolved to the
// smallest index, exactly (the tie term spans 1024 values, the distance term
// steps by 2048).  All 64 code bits are usable, the accumulator start is the
// same for every tile, and the argmin costs one integer max per distance.
// Centroid slots past C_eff in the last tile hold centroid 0 again: same
// distance, larger index, so they never win.
//
// Update step.  Member bit counts live in LDS as 16-bit pairs (dword w holds
// the counts of bits 2w and 2w+1); a lane adds its query's 32 pairs with LDS
// atomics, starting at pair (lane mod 32) so that the 64 lanes of a wave hit
// distinct dwords.  The new centroid is the per-bit majority (tie -> 0) taken
// with one wave ballot per cluster; an empty cluster keeps its code.  Integer
// arithmetic only, so the result is independent of the order of the atomics.
//
// Two drivers:
//  * kmeans_lds_kernel: one 1024-thread workgroup per (batch, head) unit for
//    n <= 4096; codes, assignments and counts stay in LDS for all L rounds,
//    only queries whose cluster changed update the counts; it writes the
//    assignments and the cluster sizes.
//  * kmeans_assign_kernel + kmeans_reduce_kernel: one launch pair per round
//    for long sequences; each 1024-query workgroup writes its partial counts
//    and a reduction kernel forms the next centroids.
#include <limits.h>

#include "common.h"
#include "hash_tile.h"
#include "kernels.h"
#include "select.h"

namespace ca {

constexpr int kCmax = 256;
constexpr int kCntStride = 33;  // dwords per cluster row of the count table (32 + 1 pad)
constexpr int kMaxQt = 16;      // query tiles of 16 per wave in both drivers

// ---------------------------------------------------------------------------
// int8 operand construction.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t spread4(uint32_t nib) {
  return (nib & 1u) | ((nib & 2u) << 7) | ((nib & 4u) << 14) | ((nib & 8u) << 21);
}

// keep[q]: byte p is 0xff when bit 16g + 4q + p is a hash bit (< n_bits);
// qslot: the query's +16 at position 63 (byte 3 of the lane group g = 3's
// last word) when that position carries the tile term (n_bits <= 63).
struct OpMasks {
  uint32_t keep[4];
  uint32_t qslot;
};
// Whether position 63 carries the tile part of the tie term.
__device__ __forceinline__ bool tile_slot(int n_bits) { return n_bits <= 63; }
__device__ __forceinline__ OpMasks op_masks(int g, int n_bits) {
  OpMasks m;
  m.qslot = (g == 3 && tile_slot(n_bits)) ? 0x10000000u : 0u;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t k = 0;
#pragma unroll
    for (int p = 0; p < 4; ++p)
      if (16 * g + 4 * q + p < n_bits) k |= 0xffu << (8 * p);
    m.keep[q] = k;
  }
  return m;
}

constexpr int kTie = 1023;  // tie term of cluster 0; cluster j has kTie - j

// Bits 16g..16g+15 of a query code as 16 int8: +64 / -64, 0 past n_bits
// (+16 at position 63 when it carries the tile term).
__device__ __forceinline__ v4i query_operand(uint64_t code, int g, const OpMasks& m) {
  const uint32_t x = static_cast<uint32_t>(code >> (16 * g)) & 0xffffu;
  v4i r;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t s = spread4((x >> (4 * q)) & 0xfu);
    r[q] = static_cast<int>((0xc0c0c0c0u ^ (s << 7)) & m.keep[q]);
  }
  r[3] |= static_cast<int>(m.qslot);
  return r;
}

// 16 code bits x (bits 16g..16g+15 of a centroid of tile ct) as 16 int8:
// +16 / -16, 0 past n_bits, and -ct at position 63 when it carries the tile
// term.
__device__ __forceinline__ v4i centroid_operand16(uint32_t x, int ct, const OpMasks& m) {
  v4i r;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t s = spread4((x >> (4 * q)) & 0xfu);
    r[q] = static_cast<int>((0xf0f0f0f0u ^ (s * 0xe0u)) & m.keep[q]);
  }
  if (m.qslot != 0u) r[3] |= static_cast<int>(static_cast<uint32_t>(-ct & 0xff) << 24);
  return r;
}
__device__ __forceinline__ v4i centroid_operand(uint64_t code, int g, int ct, const OpMasks& m) {
  return centroid_operand16(static_cast<uint32_t>(code >> (16 * g)) & 0xffffu, ct, m);
}
// Accumulator start for this lane's four result rows, centroids
// 4 (lane / 16) + i of every tile: the in-tile part of the tie term.
__device__ __forceinline__ v4i tie_start(int lane) {
  v4i r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = kTie - (4 * (lane >> 4) + i);
  return r;
}
// The largest of the lane's four keys of tile ct; SHIFT: the tile's part of
// the tie term is not in the products yet (n_bits = 64).
template <bool SHIFT>
__device__ __forceinline__ int tile_key(const v4i& d, int ct) {
  const int m = max(max(d[0], d[1]), max(d[2], d[3]));
  return SHIFT ? m - 16 * ct : m;
}

// Same as query_operand, from a table mapping 8 code bits to 8 int8 entries.
__device__ __forceinline__ v4i query_operand_lut(uint64_t code, int g, const OpMasks& m,
                                                 const uint2* lut) {
  const uint32_t x = static_cast<uint32_t>(code >> (16 * g)) & 0xffffu;
  const uint2 lo = lut[x & 0xffu], hi = lut[x >> 8];
  v4i r;
  r[0] = static_cast<int>(lo.x & m.keep[0]);
  r[1] = static_cast<int>(lo.y & m.keep[1]);
  r[2] = static_cast<int>(hi.x & m.keep[2]);
  r[3] = static_cast<int>((hi.y & m.keep[3]) | m.qslot);
  return r;
}

// Cluster index from the best key.
__device__ __forceinline__ int decode_cluster(int best, int n_bits) {
  return (1024 * n_bits + kTie - best) & 2047;
}

// Bit-pair w of a code as two 16-bit counters.
__device__ __forceinline__ uint32_t pair_val(uint64_t code, int w) {
  const uint32_t x = static_cast<uint32_t>(code >> (2 * w));
  return (x & 1u) | ((x & 2u) << 15);
}

// Best keys of NG 16-query tiles at once: one centroid-operand load feeds NG
// independent MFMAs, and the next operand is fetched before they issue.  Four
// centroid tiles are requested together (past the last tile the last one
// repeats); EXACT_TAIL takes an odd last tile alone instead of pairing it
// with a repeat, which saves its products but (measured) slows the
// one-workgroup-per-unit kernel, whose schedule favours the branch-free form.
template <int NG, bool EXACT_TAIL, bool SHIFT>
__device__ __forceinline__ void best_keys(const v4i* cop, int nct, const v4i* bq, int* best, int lane) {
  const v4i z = tie_start(lane);
  for (int ct0 = 0; ct0 < nct; ct0 += 4) {
    v4i a[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) a[q] = cop[min(ct0 + q, nct - 1) * 64 + lane];
#pragma unroll
    for (int q0 = 0; q0 < 4; q0 += 2) {  // two tiles' products in flight at a time
      if constexpr (EXACT_TAIL) {
        const int rem = nct - ct0 - q0;  // tiles left from here (uniform)
        if (rem <= 0) break;
        if (rem == 1) {
          v4i d1[NG];
#pragma unroll
          for (int e = 0; e < NG; ++e) d1[e] = mfma_i8_16x16x64(a[q0], bq[e], z);
#pragma unroll
          for (int e = 0; e < NG; ++e) best[e] = max(best[e], tile_key<SHIFT>(d1[e], ct0 + q0));
          break;
        }
      }
      v4i d[2][NG];
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int e = 0; e < NG; ++e) d[q][e] = mfma_i8_16x16x64(a[q0 + q], bq[e], z);
#pragma unroll
      for (int e = 0; e < NG; ++e)
        best[e] = max(best[e], max(tile_key<SHIFT>(d[0][e], min(ct0 + q0, nct - 1)),
                                   tile_key<SHIFT>(d[1][e], min(ct0 + q0 + 1, nct - 1))));
    }
  }
#pragma unroll
  for (int e = 0; e < NG; ++e) {
    best[e] = cross_rows_max(best[e]);
  }
}
template <bool EXACT_TAIL, bool SHIFT>
__device__ __forceinline__ void best_keys_ng(int ng, const v4i* cop, int nct, const v4i* bq,
                                             int* best, int lane) {
  switch (ng) {
    case 1: best_keys<1, EXACT_TAIL, SHIFT>(cop, nct, bq, best, lane); break;
    case 2: best_keys<2, EXACT_TAIL, SHIFT>(cop, nct, bq, best, lane); break;
    case 3: best_keys<3, EXACT_TAIL, SHIFT>(cop, nct, bq, best, lane); break;
    default: best_keys<4, EXACT_TAIL, SHIFT>(cop, nct, bq, best, lane); break;
  }
}
template <bool EXACT_TAIL>
__device__ __forceinline__ void best_keys_n(int ng, const v4i* cop, int nct, int n_bits,
                                            const v4i* bq, int* best, int lane) {
  if (tile_slot(n_bits))
    best_keys_ng<EXACT_TAIL, false>(ng, cop, nct, bq, best, lane);
  else
    best_keys_ng<EXACT_TAIL, true>(ng, cop, nct, bq, best, lane);
}

// Fills the centroid operands of nct tiles (entries e = ct * 64 + lane); the
// slots past ce hold centroid 0, whose own slot always beats them.
__device__ __forceinline__ void build_centroid_operands(v4i* cop, const uint64_t* cent, int ce,
                                                        int nct, int n_bits, int tid, int nthreads) {
  for (int e = tid; e < nct * 64; e += nthreads) {
    const int ct = e >> 6, ln = e & 63;
    const int j = ct * 16 + (ln & 15), g = ln >> 4;
    const OpMasks m = op_masks(g, n_bits);
    cop[e] = centroid_operand(cent[j < ce ? j : 0], g, ct, m);
  }
}

// ===========================================================================
// One workgroup per unit.
// ===========================================================================
constexpr int kKmThreads = 1024;
constexpr int kKmWaves = kKmThreads / 64;
static_assert(kKmLdsMaxN == kMaxQt * 16 * kKmWaves, "tile budget");

// One assign step over the n queries of a workgroup of kKmWaves waves (codes,
// assignments and counts in LDS): each query goes to the nearest centroid of
// the operand table cop (nct tiles, ce centroids), and a query whose cluster changed moves
// its bit-pair counts and its size from the old row to the new one (a first
// assignment, old = -1, only adds).  Adds the number of moved queries to
// *nchange.  bq0 / code0, when not null, are the operands and codes of each
// wave's first four query tiles, built once by the caller (otherwise every
// tile's operands come from the LDS codes).  EXACT_TAIL as in best_keys.
// Ends without a workgroup barrier.
template <bool EXACT_TAIL>
__device__ __forceinline__ void assign_round(int n, int nqt, int nct, int ce, int n_bits,
                                             const v4i* cop, const uint64_t* codes,
                                             int32_t* assign, uint32_t* cnt, int32_t* size,
                                             int* nchange, const uint2* qlut, const OpMasks& qm,
                                             const v4i* bq0, const uint64_t* code0, int lane,
                                             int wave) {
  const int g = lane >> 4, c = lane & 15;
  for (int s0 = 0; s0 < kMaxQt; s0 += 4) {
    const int left = (nqt - wave + kKmWaves - 1) / kKmWaves - s0;  // tiles of this wave not yet done
    if (left <= 0) break;
    v4i bq[4];
    int best[4];
    uint64_t mycode[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (s0 == 0 && bq0 != nullptr) {
        mycode[e] = code0[e];
        bq[e] = bq0[e];
      } else {
        const int qb = (wave + (s0 + e) * kKmWaves) * 16 + c;
        mycode[e] = qb < n ? codes[qb] : 0ull;
        bq[e] = query_operand_lut(mycode[e], g, qm, qlut);
      }
      best[e] = INT_MIN;
    }
    best_keys_n<EXACT_TAIL>(left < 4 ? left : 4, cop, nct, n_bits, bq, best, lane);
    // lane l now decides query (l % 16) of tile l / 16 of the group; the
    // queries whose cluster changed move their bit counts
    const int eq = lane >> 4;
    const int bsel = eq == 0 ? best[0] : eq == 1 ? best[1] : eq == 2 ? best[2] : best[3];
    const uint64_t code = eq == 0 ? mycode[0] : eq == 1 ? mycode[1] : eq == 2 ? mycode[2] : mycode[3];
    const int qi = (wave + (s0 + eq) * kKmWaves) * 16 + c;
    bool chg = false;
    int j = 0, old = 0;
    if (eq < left && qi < n) {
      j = decode_cluster(bsel, n_bits);
      old = assign[qi];
      chg = j != old;
      if (chg) assign[qi] = j;
    }
    const uint64_t cmask = __ballot(chg);
    const int nchg = __popcll(cmask);
    if (nchg > 32) {
      // many (the first round): every changed lane moves its own 32 words,
      // the word order rotated by lane so that the atomics spread over banks
      if (chg) {
        if (old >= 0) {
          atomicSub(&size[old], 1);
#pragma unroll 4
          for (int s = 0; s < 32; ++s) {
            const int w = (s + lane) & 31;
            atomicSub(&cnt[old * kCntStride + w], pair_val(code, w));
          }
        }
        atomicAdd(&size[j], 1);
#pragma unroll 4
        for (int s = 0; s < 32; ++s) {
          const int w = (s + lane) & 31;
          atomicAdd(&cnt[j * kCntStride + w], pair_val(code, w));
        }
      }
    } else {
      // few: one wave-wide atomic per changed query, lanes 0-31 taking its
      // words out of the old row and lanes 32-63 adding them to the new one
      uint64_t cm = cmask;
      while (cm != 0ull) {
        const int src = __ffsll(static_cast<unsigned long long>(cm)) - 1;
        cm &= cm - 1;
        const int row = lane < 32 ? __builtin_amdgcn_readlane(old, src) : __builtin_amdgcn_readlane(j, src);
        const uint64_t cs =
            (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(code >> 32), src))) << 32) |
            static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(code), src));
        const int w = lane & 31;
        const uint32_t pv = pair_val(cs, w);
        if (row >= 0) {
          atomicAdd(&cnt[row * kCntStride + w], lane < 32 ? 0u - pv : pv);
          if (w == 0) atomicAdd(&size[row], lane < 32 ? -1 : 1);
        }
      }
    }
    if (lane == 0 && nchg > 0) atomicAdd(nchange, nchg);
  }
}

// Order-preserving counting sort of the n queries of a workgroup of kKmWaves
// waves by cluster: emit(pos, i) receives every query i (assign[i] in
// [0, ce), LDS) at position off[assign[i]] + (earlier queries of that
// cluster), so that each cluster's queries come out in ascending order.  Wave
// w takes the contiguous query range [w per, (w + 1) per); within 64 queries,
// the lanes of one cluster find each other with nine ballots on the bits of
// the cluster index.  hist is LDS scratch of kKmWaves * kCmax ints, free at
// entry.  Ends without a workgroup barrier.
template <typename Emit>
__device__ __forceinline__ void member_sort(int n, int ce, const int32_t* assign, const int32_t* off,
                                            int32_t* hist, Emit emit, int tid, int lane, int wave) {
  for (int x = tid; x < kKmWaves * kCmax; x += kKmThreads) hist[x] = 0;
  const int per = (n + kKmWaves - 1) / kKmWaves;
  const int q_begin = min(n, wave * per), q_end = min(n, q_begin + per);
  auto same_cluster = [&](int a) {  // lanes whose a equals this lane's (a in [0, 511])
    uint64_t eq = ~0ull;
#pragma unroll
    for (int b = 0; b < 9; ++b) {
      const uint64_t m = __ballot((a >> b) & 1);
      eq &= ((a >> b) & 1) ? m : ~m;
    }
    return eq;
  };
  __syncthreads();
  for (int base = q_begin; base < q_end; base += 64) {
    const int i = base + lane;
    const int a = i < q_end ? assign[i] : 511;
    const uint64_t eq = same_cluster(a);
    if (a < kCmax && (eq & lanemask_lt()) == 0ull) hist[wave * kCmax + a] += __popcll(eq);
  }
  __syncthreads();
  for (int j = tid; j < ce; j += kKmThreads) {  // per-wave bases
    int run = off[j];
    for (int w = 0; w < kKmWaves; ++w) {
      const int x = hist[w * kCmax + j];
      hist[w * kCmax + j] = run;
      run += x;
    }
  }
  __syncthreads();
  for (int base = q_begin; base < q_end; base += 64) {
    const int i = base + lane;
    const int a = i < q_end ? assign[i] : 511;
    const uint64_t eq = same_cluster(a);
    if (a < kCmax) {
      const int pos = hist[wave * kCmax + a] + __popcll(eq & lanemask_lt());
      emit(pos, i);
    }
    wave_lds_sync();
    if (a < kCmax && (eq & lanemask_lt()) == 0ull) hist[wave * kCmax + a] += __popcll(eq);
    wave_lds_sync();
  }
}

struct KmShared {
  uint64_t codes[kKmLdsMaxN];
  int32_t assign[kKmLdsMaxN];
  int32_t scratch[kKmLdsMaxN];  // change list; later per-wave cluster counts
  uint32_t cnt[kCmax * kCntStride];
  int32_t size[kCmax];
  uint64_t cent[kCmax];
  v4i cop[kCmax / 16 * 64];
  uint2 qlut[256];
  int nchange[2];  // queries moved in the current round (double buffered)
};

struct FrontArgs {
  const void* q;
  const float* planes;
  const uint64_t* codes_in;  // caller-supplied codes, or null to hash
  const int32_t* lengths;
  int heads, N, C, n_bits, L;
  uint64_t* codes;    // [U][N]
  int32_t* assign;    // [U][N]
  int32_t* sizes;     // [U][C]
  int32_t* offsets;   // [U][C+1]
  int32_t* members;   // [U][N]
  float* qc;          // [U][C][D]
  void* out;          // zeroed past each sequence's length when not null
};

// One workgroup per unit runs the whole clustering: hashing (or loading the
// given codes), L K-means rounds with everything resident in LDS, the
// cluster-sorted member lists and the centroids (Eq. 3).
template <int D, typename T>
__global__ __launch_bounds__(kKmThreads) void cluster_lds_kernel(FrontArgs f) {
  __shared__ KmShared sh;
  const int u = blockIdx.x;
  const int N = f.N, C = f.C, n_bits = f.n_bits;
  const int n = unit_length(f.lengths, u / f.heads, N);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t row0 = static_cast<size_t>(u) * N;
  for (int i = n + tid; i < N; i += kKmThreads) {
    f.assign[row0 + i] = -1;
    f.codes[row0 + i] = 0;
  }
  if (f.out != nullptr) {
    T* ou = static_cast<T*>(f.out) + row0 * D;
    for (int x = n * (D / 4) + tid; x < N * (D / 4); x += kKmThreads)
      store4(ou + static_cast<size_t>(x) * 4, 0.f, 0.f, 0.f, 0.f);
  }
  if (n == 0) {
    for (int j = tid; j < C; j += kKmThreads) f.sizes[static_cast<size_t>(u) * C + j] = 0;
    for (int j = tid; j <= C; j += kKmThreads) f.offsets[static_cast<size_t>(u) * (C + 1) + j] = 0;
    for (int x = tid; x < C * D; x += kKmThreads) f.qc[static_cast<size_t>(u) * C * D + x] = 0.f;
    return;
  }
  const int ce = C < n ? C : n;
  const int nct = (ce + 15) / 16;
  const int nqt = (n + 15) / 16;
  const T* qu = static_cast<const T*>(f.q) + row0 * D;

  // ---- codes -----------------------------------------------------------------
  if (f.codes_in != nullptr) {
    const uint64_t mask = n_bits >= 64 ? ~0ull : (1ull << n_bits) - 1;
    for (int i = tid; i < n; i += kKmThreads) {
      const uint64_t x = f.codes_in[row0 + i] & mask;
      sh.codes[i] = x;
      f.codes[row0 + i] = x;
    }
  } else {
    // the planes and the waves' plane thresholds are staged in the assignment
    // and scratch areas (adjacent, both unused until the hashing ends)
    static_assert(offsetof(KmShared, scratch) == offsetof(KmShared, assign) + sizeof(sh.assign) &&
                      sizeof(sh.assign) + sizeof(sh.scratch) >=
                          (64 * kPlaneRow<D> + 64 * kKmWaves) * sizeof(float),
                  "plane staging");
    float* sp = reinterpret_cast<float*>(sh.assign);
    float* sthr = sp + 64 * kPlaneRow<D> + 64 * wave;
    const float* ph = f.planes + static_cast<size_t>(u % f.heads) * n_bits * D;
    // planes requested, then the first query tile, which stays in flight
    // while the planes go to LDS
    // (the scheduling barriers keep that order of the loads)
    PlaneStage<D, kKmThreads> stage;
    fetch_planes<D, kKmThreads>(ph, n_bits, stage, tid);
    __builtin_amdgcn_sched_barrier(0);
    const int wu = __builtin_amdgcn_readfirstlane(wave);  // uniform: the tile's buffer resource in scalars
    TileRaw<D, T> nxt = load_tile<D, T>(qu, wu * 16, wu < nqt ? min(16, n - wu * 16) : 0, lane);
    __builtin_amdgcn_sched_barrier(0);
    store_planes<D, kKmThreads>(stage, sp, tid);
    __syncthreads();
    PlaneOps<D> P;
    const bool exact_all = load_plane_ops<D>(sp, n_bits, lane, P, sthr);
    for (int tile = wu; tile < nqt; tile += kKmWaves) {
      const int r0 = tile * 16;
      const TileRaw<D, T> cur = nxt;
      const int t2 = tile + kKmWaves;
      // issued in every iteration (past the last tile it reads nothing)
      nxt = load_tile<D, T>(qu, t2 * 16, t2 < nqt ? min(16, n - t2 * 16) : 0, lane);
      const uint64_t code = hash_tile<D, T>(qu, cur, r0, min(16, n - r0), sp, n_bits, P, exact_all, lane, nullptr);
      if (lane < 16 && r0 + lane < n) {
        sh.codes[r0 + lane] = code;
        f.codes[row0 + r0 + lane] = code;
      }
    }
    __syncthreads();  // every wave is done with the staged planes
  }
  for (int i = tid; i < n; i += kKmThreads) sh.assign[i] = -1;
  for (int x = tid; x < kCmax * kCntStride; x += kKmThreads) sh.cnt[x] = 0;
  for (int j = tid; j < kCmax; j += kKmThreads) sh.size[j] = 0;
  if (tid < 2) sh.nchange[tid] = 0;
  __syncthreads();
  for (int j = tid; j < ce; j += kKmThreads)
    sh.cent[j] = sh.codes[(static_cast<int64_t>(j) * n) / ce];

  // byte pattern -> 8 int8 of +64 / -64, for rebuilding query operands cheaply
  for (int b = tid; b < 256; b += kKmThreads) {
    const uint32_t lo = 0xc0c0c0c0u ^ (spread4(b & 0xf) << 7);
    const uint32_t hi = 0xc0c0c0c0u ^ (spread4(b >> 4) << 7);
    sh.qlut[b] = make_uint2(lo, hi);
  }
  const int g = lane >> 4, c = lane & 15;
  const OpMasks qm = op_masks(g, n_bits);
  __syncthreads();

  // ---- K-means ---------------------------------------------------------------
  build_centroid_operands(sh.cop, sh.cent, ce, nct, n_bits, tid, kKmThreads);
  __syncthreads();  // the first assign step reads every centroid operand
  // operands of this wave's first four query tiles, built once: the codes
  // never change (tiles past those are rebuilt in each round)
  v4i bq0[4];
  uint64_t code0[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int qb = (wave + e * kKmWaves) * 16 + c;
    code0[e] = qb < n ? sh.codes[qb] : 0ull;
    bq0[e] = query_operand_lut(code0[e], g, qm, sh.qlut);
  }
  for (int t = 0; t < f.L; ++t) {
    // round t counts in nchange[t & 1]; the other one is cleared during this
    // round's update, after every thread has read it in the previous round
    // assign (up to four query tiles share every centroid-operand load); the
    // queries whose cluster changed move their bit counts right away
    assign_round<false>(n, nqt, nct, ce, n_bits, sh.cop, sh.codes, sh.assign, sh.cnt, sh.size,
                 &sh.nchange[t & 1], sh.qlut, qm, bq0, code0, lane, wave);
    __syncthreads();
    // no query moved: every later round would repeat this assignment
    if (sh.nchange[t & 1] == 0) break;
    if (t == f.L - 1) break;
    if (tid == 0) sh.nchange[(t + 1) & 1] = 0;
    // majority update fused with the operand rebuild: thread (tile, lane)
    // forms the 16 bits of k-group g of centroid j (slots past C_eff copy
    // centroid 0; they never win); an empty cluster keeps its operands
    for (int e = tid; e < nct * 64; e += kKmThreads) {
      const int j = (e >> 6) * 16 + c;  // e & 63 == lane because the stride is a multiple of 64
      const int src = j < ce ? j : 0;
      const int sz = sh.size[src];
      if (sz == 0) continue;
      const uint32_t* row = &sh.cnt[src * kCntStride + 8 * g];
      uint32_t bits16 = 0;
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        const uint32_t dw = row[w];
        bits16 |= static_cast<uint32_t>(2 * static_cast<int>(dw & 0xffffu) > sz) << (2 * w);
        bits16 |= static_cast<uint32_t>(2 * static_cast<int>(dw >> 16) > sz) << (2 * w + 1);
      }
      sh.cop[e] = centroid_operand16(bits16, e >> 6, qm);
    }
    __syncthreads();
  }

  // ---- member lists, ascending query order per cluster -------------------------
  int32_t* off = reinterpret_cast<int32_t*>(sh.cnt);  // [kCmax + 1], the counts are dead
  static_assert((kCmax + 8) + kKmWaves * kCmax <= kCmax * kCntStride, "member-list scratch");
  int32_t* mem = sh.scratch;
  if (wave == 0) {
    int sz4[4], local = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = 4 * lane + e;
      sz4[e] = j < ce ? sh.size[j] : 0;
      local += sz4[e];
    }
    int run = wave_incl_scan(local) - local;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      off[4 * lane + e] = run;
      run += sz4[e];
    }
    if (lane == 63) off[kCmax] = run;
  }
  __syncthreads();
  member_sort(n, ce, sh.assign, off, off + kCmax + 8, [&](int pos, int i) { mem[pos] = i; }, tid, lane, wave);
  __syncthreads();
  // ---- centroids, Eq. (3) ---------------------------------------------------------
  // D lanes (lane = dimension) per group; group g takes the sorted positions
  // [g per, (g + 1) per), all of its member rows requested together, and adds
  // them in order, one fp64 addition after the other.  A cluster that lies
  // inside the range is finished there; one cut by range ends leaves partial
  // sums in LDS (slot 0: the piece at the start of a range, slot 1: the piece
  // at its end), which the group holding the cluster's first row adds up in
  // range order after a barrier.
  constexpr int GPW = 64 / D;        // groups per wave
  constexpr int G = kKmWaves * GPW;  // groups per workgroup
  constexpr int RB = 32;             // rows in flight per lane
  double* cut = reinterpret_cast<double*>(sh.codes);  // [G][2][D]; the codes are dead
  static_assert(sizeof(sh.codes) >= static_cast<size_t>(G) * 2 * D * sizeof(double), "partial sums");
  {
    const int t = lane % D, grp = wave * GPW + lane / D;
    const int per = (n + G - 1) / G;
    const int p0 = min(n, grp * per), p1 = min(n, p0 + per);
    float* qcu = f.qc + static_cast<size_t>(u) * C * D;
    int j = 0, start = 0, end = 0;
    if (p0 < p1) {  // cluster of position p0
      j = sh.assign[mem[p0]];
      start = off[j];
      end = off[j + 1];
    }
    int s1j = -1, s1start = 0, s1end = 0;  // the cluster cut at the end of the range
    double acc = 0.0;
    for (int b0 = p0; b0 < p1; b0 += RB) {
      // positions past the range repeat its last row (straight-line loads)
      int mi[RB];
#pragma unroll
      for (int e = 0; e < RB; ++e) mi[e] = mem[min(b0 + e, p1 - 1)];
      float x[RB];
#pragma unroll
      for (int e = 0; e < RB; ++e) x[e] = to_f32(qu[static_cast<size_t>(mi[e]) * D + t]);
#pragma unroll
      for (int e = 0; e < RB; ++e) {
        const int p = b0 + e;
        if (p >= p1) continue;
        acc += static_cast<double>(x[e]);
        if (p + 1 == end) {  // cluster j ends here
          if (start >= p0) {
            qcu[j * D + t] = static_cast<float>(acc / static_cast<double>(end - start));
          } else {
            cut[(grp * 2 + 0) * D + t] = acc;
          }
          acc = 0.0;
          if (p + 1 < p1) {  // next non-empty cluster, starting at p + 1
            do {
              ++j;
              end = off[j + 1];
            } while (end == p + 1);
            start = p + 1;
          }
        } else if (p + 1 == p1) {  // the range ends inside cluster j
          if (start < p0) {
            cut[(grp * 2 + 0) * D + t] = acc;
          } else {
            cut[(grp * 2 + 1) * D + t] = acc;
            s1j = j;
            s1start = start;
            s1end = end;
          }
        }
      }
    }
    // clusters with no member, and slots past C_eff
    for (int x = tid; x < C * D; x += kKmThreads) {
      const int jj = x / D;
      if (jj >= ce || sh.size[jj] == 0) qcu[x] = 0.0f;
    }
    __syncthreads();
    if (s1j >= 0) {
      double sum = cut[(grp * 2 + 1) * D + t];
      const int g_last = (s1end - 1) / per;
      for (int gg = grp + 1; gg <= g_last; ++gg) sum += cut[(gg * 2 + 0) * D + t];
      qcu[s1j * D + t] = static_cast<float>(sum / static_cast<double>(s1end - s1start));
    }
  }
  // the clustering itself, written last so that the row loads above do not
  // wait behind these stores
  for (int i = tid; i < n; i += kKmThreads) {
    f.assign[row0 + i] = sh.assign[i];
    f.members[row0 + i] = mem[i];
  }
  for (int j = tid; j < C; j += kKmThreads) f.sizes[static_cast<size_t>(u) * C + j] = j < ce ? sh.size[j] : 0;
  for (int j = tid; j <= C; j += kKmThreads)
    f.offsets[static_cast<size_t>(u) * (C + 1) + j] = j < ce ? off[j] : n;
}

// ===========================================================================
// Cooperative path: the workgroups of a unit run all L rounds in one launch.
//
// Workgroup b of unit u holds queries [b Q, (b + 1) Q) (Q = 2048, or 1024
// when that grid does not fit on the device at once) with their codes,
// assignments and bit-pair counts resident in LDS, as the one-workgroup
// kernel does.  The unit's counts live in two running-total tables of
// 64-bit words (a cluster row has 32 words, each holding the two 32-bit
// counts of one bit pair, and its size).  In round t a workgroup adds to
// table t % 2 the change of its local counts since it last added to that
// table (two rounds earlier), as signed 64-bit atomic adds of only the words
// that changed, so that the table then holds the unit's counts of round t
// (the two halves of a word stay exact: modular arithmetic, and each final
// half is a true count).  It then waits at a per-unit arrival counter until
// every workgroup of the unit has added its part; every workgroup reads the
// whole table and forms the next centroids by the per-bit majority itself.
// Integer sums, so nothing depends on the order of the atomics.  Table t % 2
// is next changed in round t + 2, after the arrival of round t + 1, which
// every reader of round t has passed.  Arrivals go to one of two 64-bit
// words, word t % 2: each adds 1 to its low half and, when some query of the
// workgroup moved in that round, 1 to its high half.  A workgroup arrives in
// round t + 2 only after every workgroup has arrived in round t + 1, so when
// the low half of word t % 2 shows every arrival of rounds t, t - 2, ..., the
// word holds exactly those rounds' arrivals, however late the poll comes;
// its high half, against the value seen two rounds earlier, tells whether
// any query of the unit moved in round t, the same answer for every
// workgroup.  (With one word for all rounds, a poll delayed past other
// workgroups' next arrival would count their next-round moves in this round
// and could end the loop one round early in that workgroup alone.)  Every
// value that crosses workgroups travels through device-scope atomics or
// stores, each wave waits until its own have been performed before the
// workgroup barrier that precedes the arrival, and the waiting side reads
// with device-scope loads issued after it has seen every arrival; so the
// arrival itself needs no cache write-back or invalidation (which cost each
// round several microseconds when measured).  All workgroups are resident
// together, so every wait ends: the grid never exceeds what the device holds
// at once (the occupancy query times the compute units), the kernel before it
// in the stream has finished when it starts, and a waiting workgroup blocks
// no other kernel, so a workgroup held back by another stream's work is
// placed once that work drains.  (A cooperative launch gives the same
// guarantee, but measured about 15 us slower per call: it goes through a
// queue of its own.)  Each wait is also bounded.  A round in which
// no query of the unit moved ends the loop: every later round would repeat
// it.  The final member lists come from the per-workgroup sizes of the last
// round: cluster j's members of workgroup b follow those of workgroups
// 0..b-1, so each cluster's members stay in ascending query order.  When the
// grid covers every compute unit, each workgroup then adds its own members'
// rows of Q per cluster (coop_centroid_sums), so that the centroid step only
// adds the workgroups' sums; otherwise (a grid on part of the chip streams Q
// more slowly than a kernel on all of it) centroid_part_kernel forms them
// from the member ranges (bases, lsizes) written here.
// ===========================================================================
constexpr int kSpinLimit = 1 << 22;   // polls of the arrival counter before giving up
static_assert(kCoopMaxQ <= kKmLdsMaxN, "the shared assign step handles kKmLdsMaxN queries");
constexpr int kTabBatch = 8;          // table words requested together per thread
constexpr int kRowWords = 33;         // table words per cluster: 32 bit pairs and the size
static_assert(kSyncInts >= 4, "two 64-bit arrival words");

template <typename X>
__device__ __forceinline__ X ld_agent(const X* p) {
  return __hip_atomic_load(const_cast<X*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename X>
__device__ __forceinline__ void st_agent(X* p, X v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Waits until this wave's stores and atomics have been performed.
__device__ __forceinline__ void wait_memory() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

struct CoopArgs {
  const uint64_t* codes;   // [U][N]
  const int32_t* lengths;
  int heads, N, C, n_bits, L, nwg;
  int tstride;             // words per unit of a count table: C * 33
  int32_t* assign;         // [U][N]
  int32_t* sizes;          // [U][C]
  int32_t* offsets;        // [U][C+1]
  int32_t* members;        // [U][N]
  int32_t* bases;          // [U][nwg][C] first member position of (workgroup, cluster)
  int32_t* lsizes;         // [U][nwg][C] members of (workgroup, cluster)
  uint64_t* tab;           // [U][2][tstride] running count tables, zero at launch
  int32_t* sync;           // [U][kSyncInts] two 64-bit arrival words, zero at launch
  int sums;                // 1: also form the per-workgroup centroid sums
  const void* q;           // [U][N][d] queries, for the centroid sums
  int d, dtype;
  double* qc_part;         // [U][C][nwg][d] per-workgroup centroid sums
};

// Centroid sums (Eq. 3) of one workgroup of the one-launch K-means: for every
// cluster j, the fp64 sum of this workgroup's member rows of Q in ascending
// query order goes to part[(j nwg + b) d + t]; centroid_final_kernel adds the
// workgroups' sums in workgroup order and divides by the cluster size.
// Groups of D lanes (lane = dimension) take contiguous ranges of the local
// member list lmem (cluster j at positions lofs[j] .. lofs[j + 1] - 1), all of
// a range's rows requested 32 at a time and added in order; a cluster cut by
// range ends leaves partial sums in LDS (slot 0: the piece at the start of a
// range, slot 1: the piece at its end), which the group holding its first
// member adds up in range order after a barrier.  The association is fixed,
// so the result is deterministic.
template <int D, typename T>
__device__ __forceinline__ void coop_centroid_sums(const T* __restrict__ rows, const int32_t* lmem,
                                                   const int32_t* lofs, const int32_t* lassign,
                                                   const int32_t* lsize, int nq, int ce, int C,
                                                   double* cut, double* part, int nwg, int b,
                                                   int tid, int lane, int wave) {
  constexpr int GPW = 64 / D;        // groups per wave
  constexpr int G = kKmWaves * GPW;  // groups per workgroup
  constexpr int RB = 32;             // rows in flight per lane
  const int t = lane % D, grp = wave * GPW + lane / D;
  const int per = (nq + G - 1) / G;
  const int p0 = min(nq, grp * per), p1 = min(nq, p0 + per);
  auto slot = [&](int j) -> double& { return part[(static_cast<size_t>(j) * nwg + b) * D + t]; };
  int j = 0, start = 0, end = 0;
  if (p0 < p1) {  // cluster of position p0
    j = lassign[lmem[p0]];
    start = lofs[j];
    end = lofs[j + 1];
  }
  int s1j = -1, s1end = 0;  // the cluster cut at the end of the range
  double acc = 0.0;
  for (int b0 = p0; b0 < p1; b0 += RB) {
    // positions past the range repeat its last row (straight-line loads)
    int mi[RB];
#pragma unroll
    for (int e = 0; e < RB; ++e) mi[e] = lmem[min(b0 + e, p1 - 1)];
    float x[RB];
#pragma unroll
    for (int e = 0; e < RB; ++e) x[e] = to_f32(rows[static_cast<size_t>(mi[e]) * D + t]);
#pragma unroll
    for (int e = 0; e < RB; ++e) {
      const int p = b0 + e;
      if (p >= p1) continue;
      acc += static_cast<double>(x[e]);
      if (p + 1 == end) {  // cluster j ends here
        if (start >= p0)
          slot(j) = acc;
        else
          cut[(grp * 2 + 0) * D + t] = acc;
        acc = 0.0;
        if (p + 1 < p1) {  // next non-empty cluster, starting at p + 1
          do {
            ++j;
            end = lofs[j + 1];
          } while (end == p + 1);
          start = p + 1;
        }
      } else if (p + 1 == p1) {  // the range ends inside cluster j
        if (start < p0) {
          cut[(grp * 2 + 0) * D + t] = acc;
        } else {
          cut[(grp * 2 + 1) * D + t] = acc;
          s1j = j;
          s1end = end;
        }
      }
    }
  }
  // clusters with no member in this workgroup, and slots past C_eff
  for (int x = tid; x < C * D; x += kKmThreads) {
    const int jj = x / D;
    if (jj >= ce || lsize[jj] == 0) part[(static_cast<size_t>(jj) * nwg + b) * D + x % D] = 0.0;
  }
  __syncthreads();
  if (s1j >= 0) {
    double sum = cut[(grp * 2 + 1) * D + t];
    const int g_last = (s1end - 1) / per;
    for (int gg = grp + 1; gg <= g_last; ++gg) sum += cut[(gg * 2 + 0) * D + t];
    slot(s1j) = sum;
  }
}

// The 64-bit word whose even bits are e and odd bits are o.
__device__ __forceinline__ uint64_t interleave_bits(uint32_t e, uint32_t o) {
  auto spread = [](uint64_t v) {  // bit i to bit 2i
    v = (v | (v << 16)) & 0x0000ffff0000ffffull;
    v = (v | (v << 8)) & 0x00ff00ff00ff00ffull;
    v = (v | (v << 4)) & 0x0f0f0f0f0f0f0f0full;
    v = (v | (v << 2)) & 0x3333333333333333ull;
    return (v | (v << 1)) & 0x5555555555555555ull;
  };
  return spread(e) | (spread(o) << 1);
}

template <int QW>
struct CoopShared {
  uint64_t codes[QW];
  int32_t assign[QW];
  uint32_t cnt[kCmax * kCntStride];
  uint32_t pub[2][kCmax * kRowWords];  // local counts last added to each table
  int32_t size[kCmax];
  uint64_t cent[kCmax];
  v4i cop[kCmax / 16 * 64];
  uint2 qlut[256];
  int32_t tsize[kCmax];
  int32_t pre[kCmax];
  int32_t off[kCmax + 8];
  int nchange;
  int moved;  // some query of the unit moved in this round
  int ok;
};
// the member sort's per-wave counts use the operand table, dead by then
static_assert(sizeof(v4i) * (kCmax / 16 * 64) >= sizeof(int32_t) * kKmWaves * kCmax, "member-sort scratch");

// LF: the grid may hold units of exactly 65536 queries, whose narrow table
// leaves the first query out (a separate instance, so that shorter
// sequences run code without that path).
template <int QW, bool LF>
__global__ __launch_bounds__(kKmThreads) void kmeans_coop_kernel(CoopArgs a) {
  __shared__ CoopShared<QW> sh;
  const int u = blockIdx.y, b = blockIdx.x, nwg = a.nwg;
  const int N = a.N, C = a.C, n_bits = a.n_bits;
  const int n = unit_length(a.lengths, u / a.heads, N);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q0 = b * QW;
  const size_t row0 = static_cast<size_t>(u) * N;
  for (int i = max(n, q0) + tid; i < min(N, q0 + QW); i += kKmThreads) a.assign[row0 + i] = -1;
  int32_t* lsz = a.lsizes + (static_cast<size_t>(u) * nwg + b) * C;
  int32_t* bs = a.bases + (static_cast<size_t>(u) * nwg + b) * C;
  if (n == 0) {  // the same in every workgroup of the unit: none of them waits
    if (b == 0) {
      for (int j = tid; j < C; j += kKmThreads) a.sizes[static_cast<size_t>(u) * C + j] = 0;
      for (int j = tid; j <= C; j += kKmThreads) a.offsets[static_cast<size_t>(u) * (C + 1) + j] = 0;
    }
    // every block's member ranges, or its centroid sums, are empty (the
    // centroid kernels read them all)
    if (a.sums) {
      double* part = a.qc_part + static_cast<size_t>(u) * C * nwg * a.d;
      for (int x = tid; x < C * a.d; x += kKmThreads)
        part[(static_cast<size_t>(x / a.d) * nwg + b) * a.d + x % a.d] = 0.0;
    } else {
      for (int j = tid; j < C; j += kKmThreads) {
        lsz[j] = 0;
        bs[j] = 0;
      }
    }
    return;
  }
  const int nq = max(0, min(QW, n - q0));
  const int ce = C < n ? C : n;
  const int nct = (ce + 15) / 16;
  const int nqt = (nq + 15) / 16;
  const int tstride = a.tstride;
  // narrow table: 32-bit words of two 16-bit counts, half the bytes for
  // every workgroup to read each round.  For exactly 65536 queries the
  // unit's first query (held by workgroup 0) is left out of it, so that no
  // count exceeds 65535; workgroup 0 then publishes that query's cluster
  // after the table, and every reader adds the query back.
  const bool narrow = n < 65536 || (LF && n == 65536);
  const bool leave_first = LF && n == 65536;
  const uint64_t* cu = a.codes + row0;
  for (int i = tid; i < nq; i += kKmThreads) {
    sh.codes[i] = cu[q0 + i];
    sh.assign[i] = -1;
  }
  for (int x = tid; x < kCmax * kCntStride; x += kKmThreads) sh.cnt[x] = 0;
  for (int j = tid; j < kCmax; j += kKmThreads) sh.size[j] = 0;
  for (int x = tid; x < 2 * kCmax * kRowWords; x += kKmThreads) (&sh.pub[0][0])[x] = 0u;
  for (int j = tid; j < ce; j += kKmThreads) sh.cent[j] = cu[(static_cast<int64_t>(j) * n) / ce];
  for (int v = tid; v < 256; v += kKmThreads) {
    const uint32_t lo = 0xc0c0c0c0u ^ (spread4(v & 0xf) << 7);
    const uint32_t hi = 0xc0c0c0c0u ^ (spread4(v >> 4) << 7);
    sh.qlut[v] = make_uint2(lo, hi);
  }
  if (tid == 0) sh.nchange = 0;
  const OpMasks qm = op_masks(lane >> 4, n_bits);
  __syncthreads();
  build_centroid_operands(sh.cop, sh.cent, ce, nct, n_bits, tid, kKmThreads);
  __syncthreads();
  unsigned long long* arrive =
      reinterpret_cast<unsigned long long*>(a.sync + static_cast<size_t>(u) * kSyncInts);
  unsigned long long moved_seen[2] = {0, 0};  // high half of each arrival word when last seen
  for (int t = 0; t < a.L; ++t) {
    // every query tile's operands come from the LDS codes (cached operands
    // would stay live across the assign step and, with two tile groups per
    // wave, push it into spilled registers)
    assign_round<true>(nq, nqt, nct, ce, n_bits, sh.cop, sh.codes, sh.assign, sh.cnt, sh.size, &sh.nchange,
                 sh.qlut, qm, nullptr, nullptr, lane, wave);
    __syncthreads();
    // add the change of this workgroup's counts since its last addition to
    // table t % 2; keep the sizes for the member lists
    uint64_t* tab = a.tab + (static_cast<size_t>(u) * 2 + (t & 1)) * tstride;
    uint32_t* tab32 = reinterpret_cast<uint32_t*>(tab);
    uint32_t* pub = sh.pub[t & 1];
    for (int x = tid; x < ce * kRowWords; x += kKmThreads) {
      const int j = x / kRowWords, w = x - kRowWords * j;
      uint32_t cur = w < 32 ? sh.cnt[j * kCntStride + w] : static_cast<uint32_t>(sh.size[j]);
      if (leave_first && b == 0 && j == sh.assign[0]) cur -= w < 32 ? pair_val(sh.codes[0], w) : 1u;
      const uint32_t old = pub[x];
      if (cur != old && narrow) {
        // 32-bit words: the two 16-bit counts (or the size) change by the
        // difference of the packed words, modulo 2^32; once every workgroup
        // has added, the word holds the unit's counts, each below 65536
        pub[x] = cur;
        atomicAdd(&tab32[x], cur - old);
      } else if (cur != old) {
        pub[x] = cur;
        const long long dlo = static_cast<long long>(w < 32 ? (cur & 0xffffu) : cur) -
                              static_cast<long long>(w < 32 ? (old & 0xffffu) : old);
        const long long dhi = w < 32 ? static_cast<long long>(cur >> 16) - static_cast<long long>(old >> 16) : 0;
        const unsigned long long dv = static_cast<unsigned long long>(dhi) * 0x100000000ull +
                                      static_cast<unsigned long long>(dlo);
        atomicAdd(reinterpret_cast<unsigned long long*>(&tab[x]), dv);
      }
    }
    for (int j = tid; j < ce; j += kKmThreads) st_agent(&lsz[j], sh.size[j]);
    if (leave_first && b == 0 && tid == 0) st_agent(reinterpret_cast<int32_t*>(&tab32[ce * kRowWords]), sh.assign[0]);
    // arrive once every wave's additions have been performed, then wait until
    // every workgroup of the unit has arrived
    wait_memory();
    __syncthreads();
    if (tid == 0) {
      const unsigned long long add = 1ull + (sh.nchange > 0 ? 0x100000000ull : 0ull);
      sh.nchange = 0;
      unsigned long long* word = arrive + (t & 1);
      __hip_atomic_fetch_add(word, add, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // every arrival of rounds t, t - 2, ... (t / 2 + 1 per workgroup)
      const unsigned long long target = static_cast<unsigned long long>(t / 2 + 1) * nwg;
      unsigned long long seen = 0;
      int spins = 0;
      while (((seen = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) & 0xffffffffull) <
                 target &&
             spins < kSpinLimit) {
        __builtin_amdgcn_s_sleep(1);
        ++spins;
      }
      sh.ok = spins < kSpinLimit;
      const unsigned long long moves = seen >> 32;
      const unsigned long long before = (t & 1) ? moved_seen[1] : moved_seen[0];
      sh.moved = moves != before;
      if (t & 1)
        moved_seen[1] = moves;
      else
        moved_seen[0] = moves;
    }
    __syncthreads();
    if (t + 1 == a.L || !sh.moved || !sh.ok) break;  // no query moved: later rounds repeat this one
    // per-bit majority (tie -> 0) of the unit's non-empty clusters: item x
    // is pair word x % 32 of cluster x / 32 (kTabBatch words per thread in
    // flight, and lane 2e + h < 2 kTabBatch of a wave fetches the size of the
    // cluster of its half h in batch e); the 64 items of a wave are two whole
    // clusters, so two ballots give each cluster's even and odd bits, which
    // one lane per cluster interleaves into the new code
    static_assert(2 * kTabBatch <= 64, "one size per lane");
    {
      const int items = ce * 32;
      // the item index made opaque in every round, so that the loads'
      // addresses are formed here rather than kept in registers across rounds
      int tidr = tid;
      asm volatile("" : "+v"(tidr));
      for (int x0 = 0; x0 < items; x0 += kTabBatch * kKmThreads) {
        uint64_t wv[kTabBatch];
        int32_t szl = 0;
        if (narrow && !leave_first) {  // the 16-bit counts of bits 2w and 2w + 1 as the halves of a 64-bit value
#pragma unroll
          for (int e = 0; e < kTabBatch; ++e) {
            const int x = x0 + tidr + e * kKmThreads;
            const uint32_t v = x < items ? ld_agent(&tab32[(x >> 5) * kRowWords + (x & 31)]) : 0u;
            wv[e] = (v & 0xffffu) | (static_cast<uint64_t>(v >> 16) << 32);
          }
          if (lane < 2 * kTabBatch) {
            const int xs = x0 + wave * 64 + (lane & 1) * 32 + (lane >> 1) * kKmThreads;
            if (xs < items) szl = ld_agent(reinterpret_cast<const int32_t*>(&tab32[(xs >> 5) * kRowWords + 32]));
          }
        } else if (narrow) {  // the same, the first query added back to its cluster jf
          const int jf = ld_agent(reinterpret_cast<const int32_t*>(&tab32[ce * kRowWords]));
          const uint64_t cf = a.codes[row0];
          uint32_t v[kTabBatch];
#pragma unroll
          for (int e = 0; e < kTabBatch; ++e) {
            const int x = x0 + tidr + e * kKmThreads;
            v[e] = x < items ? ld_agent(&tab32[(x >> 5) * kRowWords + (x & 31)]) : 0u;
          }
          if (lane < 2 * kTabBatch) {
            const int xs = x0 + wave * 64 + (lane & 1) * 32 + (lane >> 1) * kKmThreads;
            if (xs < items) szl = ld_agent(reinterpret_cast<const int32_t*>(&tab32[(xs >> 5) * kRowWords + 32])) +
                                  ((xs >> 5) == jf ? 1 : 0);
          }
#pragma unroll
          for (int e = 0; e < kTabBatch; ++e) {
            const int x = x0 + tidr + e * kKmThreads;
            const uint32_t f = (x >> 5) == jf ? pair_val(cf, x & 31) : 0u;
            wv[e] = ((v[e] & 0xffffu) + (f & 0xffffu)) | (static_cast<uint64_t>((v[e] >> 16) + (f >> 16)) << 32);
          }
        } else {
#pragma unroll
          for (int e = 0; e < kTabBatch; ++e) {
            const int x = x0 + tidr + e * kKmThreads;
            wv[e] = x < items ? ld_agent(&tab[(x >> 5) * kRowWords + (x & 31)]) : 0ull;
          }
          // a size is a true count (at most n), so the low half of its word is it
          if (lane < 2 * kTabBatch) {
            const int xs = x0 + wave * 64 + (lane & 1) * 32 + (lane >> 1) * kKmThreads;
            if (xs < items) szl = ld_agent(reinterpret_cast<const int32_t*>(&tab[(xs >> 5) * kRowWords + 32]));
          }
        }
#pragma unroll
        for (int e = 0; e < kTabBatch; ++e) {
          const int x = x0 + tid + e * kKmThreads;
          const bool in = x < items;
          const int tz = lane < 32 ? __builtin_amdgcn_readlane(szl, 2 * e) : __builtin_amdgcn_readlane(szl, 2 * e + 1);
          const uint64_t even = __ballot(in && 2 * static_cast<long long>(wv[e] & 0xffffffffull) > tz);
          const uint64_t odd = __ballot(in && 2 * static_cast<long long>(wv[e] >> 32) > tz);
          if (in && (lane & 31) == 0 && tz > 0) {
            const int sh32 = lane & 32;  // this cluster's half of the ballots
            sh.cent[x >> 5] = interleave_bits(static_cast<uint32_t>(even >> sh32), static_cast<uint32_t>(odd >> sh32));
          }
        }
      }
    }
    __syncthreads();
    build_centroid_operands(sh.cop, sh.cent, ce, nct, n_bits, tid, kKmThreads);
    __syncthreads();
  }

  // ---- member lists from the last round's per-workgroup sizes ------------------
  // every (cluster, workgroup) size is read once, four per thread in flight:
  // the cluster's total and the part of workgroups 0..b-1
  for (int j = tid; j < ce; j += kKmThreads) sh.tsize[j] = sh.pre[j] = 0;
  __syncthreads();
  {
    const int32_t* lsu = a.lsizes + static_cast<size_t>(u) * nwg * C;
    constexpr int RB = 4;
    for (int x0 = tid; x0 < ce * nwg; x0 += RB * kKmThreads) {
      int v[RB];
#pragma unroll
      for (int e = 0; e < RB; ++e) {
        const int x = x0 + e * kKmThreads;
        v[e] = x < ce * nwg ? ld_agent(&lsu[static_cast<size_t>(x % nwg) * C + x / nwg]) : 0;
      }
#pragma unroll
      for (int e = 0; e < RB; ++e) {
        const int x = x0 + e * kKmThreads;
        if (x < ce * nwg && v[e] != 0) {
          atomicAdd(&sh.tsize[x / nwg], v[e]);
          if (x % nwg < b) atomicAdd(&sh.pre[x / nwg], v[e]);
        }
      }
    }
  }
  __syncthreads();
  // dead after the rounds: the local member list and its offsets (in the count
  // rows) and the cut sums of the centroid step (in the published counts)
  int32_t* lmem = reinterpret_cast<int32_t*>(sh.cnt);
  int32_t* lofs = lmem + QW;  // [kCmax + 1]
  double* cut = reinterpret_cast<double*>(&sh.pub[0][0]);
  static_assert(sizeof(sh.cnt) >= sizeof(int32_t) * (QW + kCmax + 1), "local member list");
  static_assert(sizeof(sh.pub) >= sizeof(double) * 2 * kKmThreads, "centroid cut sums");
  if (wave == 0) {  // exclusive scans of the unit's and this workgroup's sizes: kCmax / 64 clusters per lane
    constexpr int PL = kCmax / 64;
    int lsz4[PL], llocal = 0;
#pragma unroll
    for (int e = 0; e < PL; ++e) {
      const int j = PL * lane + e;
      lsz4[e] = j < ce ? sh.size[j] : 0;
      llocal += lsz4[e];
    }
    int lrun = wave_incl_scan(llocal) - llocal;
#pragma unroll
    for (int e = 0; e < PL; ++e) {
      lofs[PL * lane + e] = lrun;
      lrun += lsz4[e];
    }
    if (lane == 63) lofs[kCmax] = lrun;
    int sz[PL], local = 0;
#pragma unroll
    for (int e = 0; e < PL; ++e) {
      const int j = PL * lane + e;
      sz[e] = j < ce ? sh.tsize[j] : 0;
      local += sz[e];
    }
    int run = wave_incl_scan(local) - local;
#pragma unroll
    for (int e = 0; e < PL; ++e) {
      const int j = PL * lane + e;
      if (b == 0) a.offsets[static_cast<size_t>(u) * (C + 1) + min(j, C)] = j < ce ? run : n;
      sh.off[j] = run + (j < ce ? sh.pre[j] : 0);
      run += sz[e];
    }
  }
  __syncthreads();
  for (int j = tid; j < C; j += kKmThreads) {
    if (b == 0) a.sizes[static_cast<size_t>(u) * C + j] = j < ce ? sh.tsize[j] : 0;
    if (!a.sums) {  // the member ranges that centroid_part_kernel reads
      bs[j] = j < ce ? sh.off[j] : 0;
      if (j >= ce) lsz[j] = 0;
    }
  }
  if (b == 0 && tid == 0) a.offsets[static_cast<size_t>(u) * (C + 1) + C] = n;
  int32_t* mg = a.members + row0;
  member_sort(nq, ce, sh.assign, sh.off, reinterpret_cast<int32_t*>(sh.cop),
              [&](int pos, int i) {
                mg[pos] = q0 + i;
                if (a.sums) {
                  const int j = sh.assign[i];
                  lmem[lofs[j] + pos - sh.off[j]] = i;
                }
              },
              tid, lane, wave);
  if (!a.sums) {
    for (int i = tid; i < nq; i += kKmThreads) a.assign[row0 + q0 + i] = sh.assign[i];
    return;  // uniform over the workgroup
  }
  __syncthreads();
  double* part = a.qc_part + static_cast<size_t>(u) * C * nwg * a.d;
  const size_t rbase = (row0 + q0) * static_cast<size_t>(a.d);
  if (a.d == 64) {
    if (a.dtype == 0)
      coop_centroid_sums<64>(static_cast<const float*>(a.q) + rbase, lmem, lofs, sh.assign, sh.size, nq, ce, C,
                             cut, part, nwg, b, tid, lane, wave);
    else
      coop_centroid_sums<64>(static_cast<const bf16_t*>(a.q) + rbase, lmem, lofs, sh.assign, sh.size, nq, ce,
                             C, cut, part, nwg, b, tid, lane, wave);
  } else {
    if (a.dtype == 0)
      coop_centroid_sums<32>(static_cast<const float*>(a.q) + rbase, lmem, lofs, sh.assign, sh.size, nq, ce, C,
                             cut, part, nwg, b, tid, lane, wave);
    else
      coop_centroid_sums<32>(static_cast<const bf16_t*>(a.q) + rbase, lmem, lofs, sh.assign, sh.size, nq, ce,
                             C, cut, part, nwg, b, tid, lane, wave);
  }
  // the assignment, written last so that the row loads above do not wait
  // behind these stores
  for (int i = tid; i < nq; i += kKmThreads) a.assign[row0 + q0 + i] = sh.assign[i];
}

// ===========================================================================
// Multi-workgroup path: one launch pair per Lloyd round.
// ===========================================================================
constexpr int kKbThreads = 512;
constexpr int kKbWaves = kKbThreads / 64;
static_assert(kKmBlockQ <= kMaxQt * 16 * kKbWaves, "tile budget");

__global__ __launch_bounds__(kKbThreads) void kmeans_assign_kernel(
    const uint64_t* __restrict__ codes_g, const int32_t* __restrict__ lengths, int heads, int N,
    int C, int n_bits, int t, uint64_t* __restrict__ cent_cur, int32_t* __restrict__ assign_g,
    uint32_t* __restrict__ part, int32_t* __restrict__ part_sizes, int nblk) {
  __shared__ uint64_t cent[kCmax];
  __shared__ v4i cop[kCmax / 16 * 64];
  __shared__ uint32_t cnt[kCmax * kCntStride];
  __shared__ int32_t size[kCmax];
  __shared__ int32_t la[kKmBlockQ];
  __shared__ uint64_t lcodes[kKmBlockQ];
  const int u = blockIdx.y, blk = blockIdx.x;
  const int n = unit_length(lengths, u / heads, N);
  const int q0 = blk * kKmBlockQ;
  if (q0 >= n) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nq = min(kKmBlockQ, n - q0);
  const int ce = C < n ? C : n;
  const int nct = (ce + 15) / 16;
  const uint64_t* cu = codes_g + static_cast<size_t>(u) * N;
  for (int j = tid; j < ce; j += kKbThreads) {
    const uint64_t cj = t == 0 ? cu[(static_cast<int64_t>(j) * n) / ce]
                               : cent_cur[static_cast<size_t>(u) * C + j];
    cent[j] = cj;
    if (t == 0 && blk == 0) cent_cur[static_cast<size_t>(u) * C + j] = cj;
  }
  for (int x = tid; x < nq; x += kKbThreads) lcodes[x] = cu[q0 + x];
  for (int x = tid; x < kCmax * kCntStride; x += kKbThreads) cnt[x] = 0;
  for (int j = tid; j < kCmax; j += kKbThreads) size[j] = 0;
  __syncthreads();
  build_centroid_operands(cop, cent, ce, nct, n_bits, tid, kKbThreads);
  __syncthreads();
  const int g = lane >> 4, c = lane & 15;
  const OpMasks qm = op_masks(g, n_bits);
  const int nqt = (nq + 15) / 16;
  for (int s0 = 0; s0 < kMaxQt; s0 += 4) {
    const int left = (nqt - wave + kKbWaves - 1) / kKbWaves - s0;
    if (left <= 0) break;
    v4i bq[4];
    int best[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int qi = (wave + (s0 + e) * kKbWaves) * 16 + c;
      bq[e] = query_operand(qi < nq ? lcodes[qi] : 0ull, g, qm);
      best[e] = INT_MIN;
    }
    best_keys_n<true>(left < 4 ? left : 4, cop, nct, n_bits, bq, best, lane);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int qo = (wave + (s0 + e) * kKbWaves) * 16 + lane;
      if (lane < 16 && qo < nq) {
        const int j = decode_cluster(best[e], n_bits);
        la[qo] = j;
        assign_g[static_cast<size_t>(u) * N + q0 + qo] = j;
      }
    }
  }
  __syncthreads();
  for (int x = tid; x < nq; x += kKbThreads) {
    const int a = la[x];
    const uint64_t code = lcodes[x];
    atomicAdd(&size[a], 1);
#pragma unroll 4
    for (int s = 0; s < 32; ++s) {
      const int w = (s + lane) & 31;
      atomicAdd(&cnt[a * kCntStride + w], pair_val(code, w));
    }
  }
  __syncthreads();
  const size_t base = (static_cast<size_t>(u) * nblk + blk) * C;
  for (int x = tid; x < ce * 32; x += kKbThreads) {
    const int j = x >> 5, w = x & 31;
    part[(base + j) * 32 + w] = cnt[j * kCntStride + w];
  }
  for (int j = tid; j < ce; j += kKbThreads) part_sizes[base + j] = size[j];
}

// One wave per cluster: sums the partial counts and forms the next centroid.
__global__ __launch_bounds__(256) void kmeans_reduce_kernel(
    const uint32_t* __restrict__ part, const int32_t* __restrict__ part_sizes,
    const int32_t* __restrict__ lengths, int heads, int N, int C, int nblk,
    const uint64_t* __restrict__ cent_cur, uint64_t* __restrict__ cent_next) {
  const int u = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = blockIdx.x * 4 + wave;
  const int n = unit_length(lengths, u / heads, N);
  const int ce = C < n ? C : n;
  if (j >= ce) return;
  const int nb = (n + kKmBlockQ - 1) / kKmBlockQ;
  int cnt = 0, sz = 0;
  // eight blocks' partials requested at a time (integer sums: any order)
  constexpr int RB = 8;
  for (int b0 = 0; b0 < nb; b0 += RB) {
    uint32_t dw[RB];
    int ps[RB];
#pragma unroll
    for (int e = 0; e < RB; ++e) {
      const int blk = min(b0 + e, nb - 1);
      const size_t base = (static_cast<size_t>(u) * nblk + blk) * C + j;
      dw[e] = part[base * 32 + (lane >> 1)];
      ps[e] = part_sizes[base];
    }
#pragma unroll
    for (int e = 0; e < RB; ++e) {
      if (b0 + e < nb) {
        cnt += static_cast<int>((dw[e] >> ((lane & 1) * 16)) & 0xffffu);
        sz += ps[e];
      }
    }
  }
  const uint64_t bits = __ballot(2 * cnt > sz);
  if (lane == 0)
    cent_next[static_cast<size_t>(u) * C + j] = sz > 0 ? bits : cent_cur[static_cast<size_t>(u) * C + j];
}

// ===========================================================================
// CSR build from an assignment array (multi-workgroup path and injected
// assignments): per-block counts, prefix over blocks and clusters, stable
// scatter.  Assignments outside [0, C_eff) are clamped into it.
// ===========================================================================
__device__ __forceinline__ int clamp_cluster(int a, int ce) {
  return a < 0 ? 0 : (a >= ce ? ce - 1 : a);
}

__global__ __launch_bounds__(kCsrBlockQ) void csr_count_kernel(
    const int32_t* __restrict__ assign, const int32_t* __restrict__ lengths, int heads, int N,
    int C, int ncsr, int32_t* __restrict__ csr_cnt, int32_t* __restrict__ assign_pad) {
  __shared__ int32_t cnt[kCmax];
  const int u = blockIdx.y, blk = blockIdx.x, tid = threadIdx.x;
  const int n = unit_length(lengths, u / heads, N);
  const int ce = C < n ? C : n;
  const int i = blk * kCsrBlockQ + tid;
  if (assign_pad != nullptr && i >= n && i < N) assign_pad[static_cast<size_t>(u) * N + i] = -1;
  if (blk * kCsrBlockQ >= n) return;
  for (int j = tid; j < C; j += kCsrBlockQ) cnt[j] = 0;
  __syncthreads();
  if (i < n) atomicAdd(&cnt[clamp_cluster(assign[static_cast<size_t>(u) * N + i], ce)], 1);
  __syncthreads();
  for (int j = tid; j < C; j += kCsrBlockQ) csr_cnt[(static_cast<size_t>(u) * ncsr + blk) * C + j] = cnt[j];
}

__global__ __launch_bounds__(256) void csr_scan_kernel(int32_t* __restrict__ csr_cnt,
                                                       const int32_t* __restrict__ lengths, int heads,
                                                       int N, int C, int ncsr,
                                                       int32_t* __restrict__ sizes,
                                                       int32_t* __restrict__ offsets) {
  __shared__ int32_t wtot[4];
  const int u = blockIdx.x, j = threadIdx.x, lane = j & 63, wave = j >> 6;
  const int n = unit_length(lengths, u / heads, N);
  const int nb = (n + kCsrBlockQ - 1) / kCsrBlockQ;
  int run = 0;
  if (j < C) {
    // exclusive prefix over the blocks, sixteen block counts requested at a time
    constexpr int RB = 16;
    for (int b0 = 0; b0 < nb; b0 += RB) {
      int v[RB];
#pragma unroll
      for (int e = 0; e < RB; ++e)
        v[e] = b0 + e < nb ? csr_cnt[(static_cast<size_t>(u) * ncsr + b0 + e) * C + j] : 0;
#pragma unroll
      for (int e = 0; e < RB; ++e) {
        if (b0 + e < nb) csr_cnt[(static_cast<size_t>(u) * ncsr + b0 + e) * C + j] = run;
        run += v[e];
      }
    }
  }
  const int incl = wave_incl_scan(run);
  if (lane == 63) wtot[wave] = incl;
  __syncthreads();
  int excl = incl - run;
  for (int w = 0; w < wave; ++w) excl += wtot[w];
  if (j < C) {
    sizes[static_cast<size_t>(u) * C + j] = run;
    offsets[static_cast<size_t>(u) * (C + 1) + j] = excl;
    if (j == C - 1) offsets[static_cast<size_t>(u) * (C + 1) + C] = excl + run;
    for (int blk = 0; blk < nb; ++blk) csr_cnt[(static_cast<size_t>(u) * ncsr + blk) * C + j] += excl;
  }
}

__global__ __launch_bounds__(kCsrBlockQ) void csr_scatter_kernel(
    const int32_t* __restrict__ assign, const int32_t* __restrict__ lengths, int heads, int N,
    int C, int ncsr, const int32_t* __restrict__ csr_base, int32_t* __restrict__ members) {
  __shared__ int32_t wcnt[kCsrBlockQ / 64][kCmax];
  const int u = blockIdx.y, blk = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = unit_length(lengths, u / heads, N);
  if (blk * kCsrBlockQ >= n) return;
  const int ce = C < n ? C : n;
  const int i = blk * kCsrBlockQ + tid;
  const int a = i < n ? clamp_cluster(assign[static_cast<size_t>(u) * N + i], ce) : -1;
  for (int x = tid; x < (kCsrBlockQ / 64) * kCmax; x += kCsrBlockQ) (&wcnt[0][0])[x] = 0;
  __syncthreads();
  uint64_t active = __ballot(a >= 0);
  int rank = 0;
  while (active) {
    const int leader = __ffsll(static_cast<unsigned long long>(active)) - 1;
    const int aj = __builtin_amdgcn_readlane(a, leader);
    const uint64_t mm = __ballot(a == aj) & active;
    if (a == aj) rank = __popcll(mm & lanemask_lt());
    if (lane == leader) wcnt[wave][aj] = __popcll(mm);
    active &= ~mm;
  }
  __syncthreads();
  if (a >= 0) {
    int base = csr_base[(static_cast<size_t>(u) * ncsr + blk) * C + a];
    for (int w = 0; w < wave; ++w) base += wcnt[w][a];
    members[static_cast<size_t>(u) * N + base + rank] = i;
  }
}

// Copies caller-supplied assignments, clamped into [0, C_eff), -1 on padded rows.
__global__ __launch_bounds__(256) void load_assign_kernel(const int32_t* __restrict__ in,
                                                          const int32_t* __restrict__ lengths,
                                                          int heads, int N, int C,
                                                          int32_t* __restrict__ assign) {
  const int u = blockIdx.y;
  const int n = unit_length(lengths, u / heads, N);
  const int ce = C < n ? C : n;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= N) return;
  const size_t x = static_cast<size_t>(u) * N + i;
  assign[x] = i < n ? clamp_cluster(in[x], ce) : -1;
}

// ===========================================================================
// Host launchers.
// ===========================================================================
static int g_kmeans_path = 0;
void set_kmeans_path(int path) { g_kmeans_path = path; }

// Workgroups of the cooperative K-means (QW queries each) that the current
// device holds at once (its occupancy times the compute units), measured once
// per device.
template <int QW, bool LF>
static int coop_capacity_of() {
  constexpr int kMaxDev = 64;
  static int cap[kMaxDev] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) return 0;
  if (cap[dev] == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kmeans_coop_kernel<QW, LF>, kKmThreads, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cap[dev] = per_cu * cus > 0 ? per_cu * cus : -1;
  }
  return cap[dev] > 0 ? cap[dev] : 0;
}
// Workgroups that both instances of a query-block size can hold at once.
template <int QW>
static int coop_capacity() {
  return min(coop_capacity_of<QW, false>(), coop_capacity_of<QW, true>());
}

int coop_fused_sums(const Problem& p, int coop_q) {
  if (coop_q <= 0 || g_kmeans_path == 5) return 0;
  if (g_kmeans_path == 4) return 1;
  constexpr int kMaxDev = 64;
  static int cus[kMaxDev] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) return 0;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cus[dev] = n > 0 ? n : -1;
  }
  const long long wgs = static_cast<long long>(p.units()) * ((p.n + coop_q - 1) / coop_q);
  return cus[dev] > 0 && wgs >= cus[dev] ? 1 : 0;
}

int coop_block_queries(const Problem& p, int max_blocks) {
  const long long U = p.units();
  auto fits = [&](int qw, int cap) {
    const long long nb = (p.n + qw - 1) / qw;
    return nb <= max_blocks && nb * U <= cap;
  };
  if (fits(2048, coop_capacity<2048>())) return 2048;
  if (fits(1024, coop_capacity<1024>())) return 1024;
  return 0;
}

static bool coop_fits(const Problem& p) {
  return coop_block_queries(p, coop_max_blocks(p.n, p.units())) > 0;
}

int kmeans_driver(const Problem& p) {
  if (g_kmeans_path == 1 && p.n <= kKmLdsMaxN) return 1;
  if (g_kmeans_path == 2) return 2;
  if (g_kmeans_path >= 3) return coop_fits(p) ? 3 : 2;
  if (kmeans_uses_lds(p)) return 1;
  return coop_fits(p) ? 3 : 2;
}

int kmeans_uses_lds(const Problem& p) {
  if (p.n > kKmLdsMaxN) return 0;
  if (g_kmeans_path == 1) return 1;
  if (g_kmeans_path == 2) return 0;
  // One workgroup per unit when there are enough units to occupy the chip
  // or the sequences are short; otherwise spread each unit over workgroups
  // (its chain of per-round launches costs about 0.25 ms, which a single
  // workgroup per unit beats up to n = 2048 even with 8 units).
  return (p.units() >= 128 || p.n <= 2048) ? 1 : 0;
}

hipError_t launch_load_assign(const Problem& p, const int32_t* assign_in, const Workspace& ws,
                              hipStream_t s) {
  hipLaunchKernelGGL(load_assign_kernel, dim3((p.n + 255) / 256, p.units()), dim3(256), 0, s,
                     assign_in, p.lengths, p.heads, p.n, p.C, ws.assign);
  return hipGetLastError();
}

hipError_t launch_csr(const Problem& p, const int32_t* assign, const Workspace& ws, hipStream_t s) {
  const int U = p.units();
  dim3 grid(ws.ncsr, U);
  int32_t* pad = (assign == ws.assign) ? ws.assign : nullptr;
  hipLaunchKernelGGL(csr_count_kernel, grid, dim3(kCsrBlockQ), 0, s, assign, p.lengths, p.heads,
                     p.n, p.C, ws.ncsr, ws.csr_cnt, pad);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(csr_scan_kernel, dim3(U), dim3(256), 0, s, ws.csr_cnt, p.lengths, p.heads,
                     p.n, p.C, ws.ncsr, ws.sizes, ws.offsets);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(csr_scatter_kernel, grid, dim3(kCsrBlockQ), 0, s, assign, p.lengths, p.heads,
                     p.n, p.C, ws.ncsr, ws.csr_cnt, ws.members);
  return hipGetLastError();
}

template <int D, typename T>
static hipError_t launch_cluster_lds_t(const Problem& p, const uint64_t* codes_in,
                                       const Workspace& ws, hipStream_t s) {
  FrontArgs f;
  f.q = p.q;
  f.planes = p.planes;
  f.codes_in = codes_in;
  f.lengths = p.lengths;
  f.heads = p.heads;
  f.N = p.n;
  f.C = p.C;
  f.n_bits = p.n_bits;
  f.L = p.L;
  f.codes = ws.codes;
  f.assign = ws.assign;
  f.sizes = ws.sizes;
  f.offsets = ws.offsets;
  f.members = ws.members;
  f.qc = ws.qc;
  f.out = p.lengths ? p.out : nullptr;
  hipLaunchKernelGGL((cluster_lds_kernel<D, T>), dim3(p.units()), dim3(kKmThreads), 0, s, f);
  return hipGetLastError();
}

hipError_t launch_cluster_lds(const Problem& p, const uint64_t* codes_in, const Workspace& ws,
                              hipStream_t s) {
  if (p.d == 32)
    return p.dtype == 0 ? launch_cluster_lds_t<32, float>(p, codes_in, ws, s)
                        : launch_cluster_lds_t<32, bf16_t>(p, codes_in, ws, s);
  return p.dtype == 0 ? launch_cluster_lds_t<64, float>(p, codes_in, ws, s)
                      : launch_cluster_lds_t<64, bf16_t>(p, codes_in, ws, s);
}

int coop_table_stride(int C) { return C * kRowWords; }

hipError_t launch_kmeans_coop(const Problem& p, const Workspace& ws, hipStream_t s) {
  CoopArgs a;
  a.codes = ws.codes;
  a.lengths = p.lengths;
  a.heads = p.heads;
  a.N = p.n;
  a.C = p.C;
  a.n_bits = p.n_bits;
  a.L = p.L;
  a.nwg = (p.n + ws.coop_q - 1) / ws.coop_q;
  a.tstride = coop_table_stride(p.C);
  a.assign = ws.assign;
  a.sizes = ws.sizes;
  a.offsets = ws.offsets;
  a.members = ws.members;
  a.lsizes = ws.clsizes;
  a.tab = ws.ctab;
  a.sync = ws.sync;
  a.bases = ws.cbases;
  a.sums = ws.coop_sums;
  a.q = p.q;
  a.d = p.d;
  a.dtype = p.dtype;
  a.qc_part = ws.qc_part;
  void* args[] = {&a};
  const dim3 grid(a.nwg, p.units());
  const bool lf = p.n >= 65536;  // some unit may hold exactly 65536 queries
  const void* fn = nullptr;
  switch (ws.coop_q) {
    case 1024:
      fn = lf ? reinterpret_cast<const void*>(kmeans_coop_kernel<1024, true>)
              : reinterpret_cast<const void*>(kmeans_coop_kernel<1024, false>);
      break;
    case 2048:
      fn = lf ? reinterpret_cast<const void*>(kmeans_coop_kernel<2048, true>)
              : reinterpret_cast<const void*>(kmeans_coop_kernel<2048, false>);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipLaunchKernel(fn, grid, dim3(kKmThreads), args, 0, s);
}

hipError_t launch_kmeans(const Problem& p, const Workspace& ws, hipStream_t s) {
  const int U = p.units();
  uint64_t* cent0 = ws.cent;
  uint64_t* cent1 = ws.cent + static_cast<size_t>(U) * p.C;
  for (int t = 0; t < p.L; ++t) {
    uint64_t* cur = (t & 1) ? cent1 : cent0;
    uint64_t* nxt = (t & 1) ? cent0 : cent1;
    hipLaunchKernelGGL(kmeans_assign_kernel, dim3(ws.nblk, U), dim3(kKbThreads), 0, s, ws.codes,
                       p.lengths, p.heads, p.n, p.C, p.n_bits, t, cur, ws.assign, ws.part,
                       ws.part_sizes, ws.nblk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (t + 1 < p.L) {
      hipLaunchKernelGGL(kmeans_reduce_kernel, dim3((p.C + 3) / 4, U), dim3(256), 0, s, ws.part,
                         ws.part_sizes, p.lengths, p.heads, p.n, p.C, ws.nblk, cur, nxt);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

}  // namespace ca
