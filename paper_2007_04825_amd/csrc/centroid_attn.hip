// Centroids (Eq. 3), centroid attention (Eqs. 4-5), the top-k keys of each
// cluster with their attention mass (Section 3.3) and the per-query outputs
// (Eq. 6 or the improved values).
//
// centroid_kernel: one wave per cluster sums the member rows of Q in fp64
//   (members in ascending query order) and divides by the cluster size (the
//   single-workgroup clustering kernel forms its centroids itself).
//
// attn_tile_kernel: one workgroup of eight waves per (unit, 16 centroids,
//   1024-key chunk).  Logits S^T = K Q^c^T come from v_mfma_f32_16x16x4f32
//   with keys as rows and centroids as columns, scaled by 1/sqrt(d), masked
//   past the valid length and kept in LDS (A^c is never written to memory);
//   while they sit in the result registers every lane also keeps the maximum
//   and, for the improved variant, the four largest logits of its slice of
//   the row.  Two rows per wave (one 32-lane group each) then take the row
//   maximum m from the slice maxima and, for the improved variant, the top-k
//   set: a threshold from the slices' kept logits, one sweep for the
//   positions that reach it.  V^T P^T accumulates the values on the matrix
//   cores: the result registers of the first product are in the B-operand
//   layout of the second (key 4g+i of a tile sits in lane group g, register
//   i), so P never leaves registers.
//   * single chunk (n <= 1024): the workgroup finishes the clusters.  The
//     clustered variant writes V^c to every member row (Eq. 6).  For the
//     improved variant the top-k keys are masked out of P, so the product
//     yields the rest part V^b = sum_{l not in T} A^c_l V_l directly, and
//     m_j = sum_{l in T} A^c_l; sparse_kernel then writes the member rows.
//   * several chunks: it writes (m, z, unnormalised values, top-k candidates)
//     of its chunk; attn_merge_kernel combines the chunks (log-sum-exp rule),
//     selects T among the candidates and forms m_j and V^b = V^c - sum_T A^c V.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "select.h"

namespace ca {

// ---------------------------------------------------------------------------
// Eq. (3)
// ---------------------------------------------------------------------------
template <int D, typename T>
__global__ __launch_bounds__(256) void centroid_kernel(const T* __restrict__ q,
                                                       const int32_t* __restrict__ sizes,
                                                       const int32_t* __restrict__ offsets,
                                                       const int32_t* __restrict__ members,
                                                       int N, int C, float* __restrict__ qc) {
  // D lanes per cluster (lane = dimension) add the member rows in ascending
  // query order, one fp64 addition after the other, eight rows in flight
  constexpr int GPW = 64 / D;  // clusters per wave
  const int u = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = (blockIdx.x * 4 + wave) * GPW + lane / D;
  const int t = lane % D;
  if (j >= C) return;
  const int sz = sizes[static_cast<size_t>(u) * C + j];
  float* dst = qc + (static_cast<size_t>(u) * C + j) * D;
  if (sz == 0) {
    dst[t] = 0.0f;
    return;
  }
  const int32_t* mem = members + static_cast<size_t>(u) * N + offsets[static_cast<size_t>(u) * (C + 1) + j];
  const T* qu = q + static_cast<size_t>(u) * N * D;
  double acc = 0.0;
  int m = 0;
  // 32 member rows in flight, their indices requested one batch ahead
  constexpr int RB = 32;
  int mi[RB];
#pragma unroll
  for (int e = 0; e < RB; ++e) mi[e] = mem[min(e, sz - 1)];
  for (; m + RB <= sz; m += RB) {
    float x[RB];
#pragma unroll
    for (int e = 0; e < RB; ++e) x[e] = to_f32(qu[static_cast<size_t>(mi[e]) * D + t]);
#pragma unroll
    for (int e = 0; e < RB; ++e) mi[e] = mem[min(m + RB + e, sz - 1)];
#pragma unroll
    for (int e = 0; e < RB; ++e) acc += static_cast<double>(x[e]);
  }
  if (m < sz) {  // the rest, whose indices are in mi already: every row requested, then added in order
    float x[RB];
#pragma unroll
    for (int e = 0; e < RB; ++e) x[e] = to_f32(qu[static_cast<size_t>(mi[e]) * D + t]);
#pragma unroll
    for (int e = 0; e < RB; ++e)
      if (m + e < sz) acc += static_cast<double>(x[e]);
  }
  dst[t] = static_cast<float>(acc / static_cast<double>(sz));
}

// Eq. (3) after the cooperative K-means, in two steps.  Step 1 (unless the
// K-means kernel formed these sums itself): for every (unit, block of coop_q
// queries, cluster) D / VL lanes add the block's members of the cluster
// (consecutive in the member list, ascending query order) in fp64, VL
// dimensions per lane: with VL = 4 a wave takes 256 / D such items at once,
// 16 rows in flight (for grids of many items); with VL = 1, 64 / D items,
// 32 rows in flight.  Step 2: the blocks' sums are added in block order and
// divided by the cluster size.  The association is fixed, so the result is
// deterministic.
template <int D, typename T, int VL>
__global__ __launch_bounds__(256) void centroid_part_kernel(const T* __restrict__ q,
                                                            const int32_t* __restrict__ members,
                                                            const int32_t* __restrict__ bases,
                                                            const int32_t* __restrict__ lsizes,
                                                            int N, int C, int nwg, long long nitems,
                                                            double* __restrict__ qc_part) {
  static_assert(VL == 1 || VL == 4, "dimensions per lane");
  constexpr int LPI = D / VL;     // lanes per item
  constexpr int GPW = 64 / LPI;   // items per wave
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long long item = (static_cast<long long>(blockIdx.x) * 4 + wave) * GPW + lane / LPI;
  const int t0 = VL * (lane % LPI);
  if (item >= nitems) return;  // item = (u nwg + b) C + j, the layout of bases and lsizes
  const int j = static_cast<int>(item % C);
  const long long ub = item / C;
  const int b = static_cast<int>(ub % nwg);
  const int u = static_cast<int>(ub / nwg);
  const int cnt = lsizes[item];
  const int32_t* mem = members + static_cast<size_t>(u) * N + bases[item];
  const T* qu = q + static_cast<size_t>(u) * N * D + t0;
  double acc[VL];
#pragma unroll
  for (int v = 0; v < VL; ++v) acc[v] = 0.0;
  constexpr int RB = VL == 4 ? 16 : 32;
  for (int m = 0; m < cnt; m += RB) {
    int mi[RB];
#pragma unroll
    for (int e = 0; e < RB; ++e) mi[e] = mem[min(m + e, cnt - 1)];
    float x[RB][VL];
#pragma unroll
    for (int e = 0; e < RB; ++e) {
      if constexpr (VL == 4)
        load4(qu + static_cast<size_t>(mi[e]) * D, x[e]);
      else
        x[e][0] = to_f32(qu[static_cast<size_t>(mi[e]) * D]);
    }
#pragma unroll
    for (int e = 0; e < RB; ++e)
      if (m + e < cnt) {
#pragma unroll
        for (int v = 0; v < VL; ++v) acc[v] += static_cast<double>(x[e][v]);
      }
  }
  double* dst = qc_part + ((static_cast<size_t>(u) * C + j) * nwg + b) * D + t0;
#pragma unroll
  for (int v = 0; v < VL; ++v) dst[v] = acc[v];
}

template <int D>
__global__ __launch_bounds__(256) void centroid_final_kernel(const double* __restrict__ qc_part,
                                                             const int32_t* __restrict__ sizes,
                                                             int C, int nwg, long long nitems,
                                                             float* __restrict__ qc) {
  constexpr int GPW = 64 / D;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long long item = (static_cast<long long>(blockIdx.x) * 4 + wave) * GPW + lane / D;  // u C + j
  const int t = lane % D;
  if (item >= nitems) return;
  const int sz = sizes[item];
  const double* pp = qc_part + static_cast<size_t>(item) * nwg * D + t;
  // the parts in block order, eight loads in flight ahead of the additions
  double acc = 0.0;
  int b = 0;
  for (; b + 8 <= nwg; b += 8) {
    double x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = pp[static_cast<size_t>(b + e) * D];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += x[e];
  }
  for (; b < nwg; ++b) acc += pp[static_cast<size_t>(b) * D];
  qc[static_cast<size_t>(item) * D + t] = sz > 0 ? static_cast<float>(acc / static_cast<double>(sz)) : 0.0f;
}

// ---------------------------------------------------------------------------
// Small vector helpers for the DT-wide value loads.
// ---------------------------------------------------------------------------
template <int W>
__device__ __forceinline__ void load_vec(const float* p, float* d) {
  if constexpr (W == 4) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    d[0] = t.x; d[1] = t.y; d[2] = t.z; d[3] = t.w;
  } else {
    const float2 t = *reinterpret_cast<const float2*>(p);
    d[0] = t.x; d[1] = t.y;
  }
}
template <int W>
__device__ __forceinline__ void load_vec(const bf16_t* p, float* d) {
  if constexpr (W == 4) {
    const uint2 t = *reinterpret_cast<const uint2*>(p);
    d[0] = __uint_as_float(t.x << 16); d[1] = __uint_as_float(t.x & 0xffff0000u);
    d[2] = __uint_as_float(t.y << 16); d[3] = __uint_as_float(t.y & 0xffff0000u);
  } else {
    const uint32_t t = *reinterpret_cast<const uint32_t*>(p);
    d[0] = __uint_as_float(t << 16); d[1] = __uint_as_float(t & 0xffff0000u);
  }
}
// Stores W consecutive fp32 values as the output type.
template <int W>
__device__ __forceinline__ void store_vec(float* p, const float* s) {
#pragma unroll
  for (int i = 0; i < W; i += 4) store4(p + i, s[i], s[i + 1], s[i + 2], s[i + 3]);
}
template <int W>
__device__ __forceinline__ void store_vec(bf16_t* p, const float* s) {
#pragma unroll
  for (int i = 0; i < W; i += 4) store4(p + i, s[i], s[i + 1], s[i + 2], s[i + 3]);
}

// ---------------------------------------------------------------------------
// Centroid attention tile kernel.
// ---------------------------------------------------------------------------
// Floats per LDS logit row: a stride of 4 mod 64 puts the float4 accesses of
// the 16 rows (lane c = row, lane group g = keys 4g..4g+3 of a tile) in
// distinct banks.
constexpr int kLStride = kChunk + 4;
static_assert(kLStride >= kChunk, "rows padded for the top-k sweep: 32 grp_block_len(kChunk) <= kChunk");
constexpr int kRedPad = 4;  // floats of padding per row of the cross-wave reduction
constexpr int kCandCap = 128;
// Whether fp32 inputs take the centroid products on the bf16 matrix cores
// with both operands split in three (six part products, fp32 accuracy)
// instead of the fp32 matrix cores.  The bf16 instruction does eight times
// the work of v_mfma_f32_16x16x4f32 in half the cycles, but measured on the
// length-sweep point N = 32768 the single-pass kernel ran no faster (it is
// not bound by the matrix cores) and the tile kernel slower (the splits cost
// registers: 169 instead of one workgroup's worth of occupancy), so fp32
// keeps the fp32 matrix cores.
constexpr bool kSplitF32 = false;
constexpr int kSparseChunk = 64;  // members per work item of sparse_kernel
constexpr int kTileWaves = 8;  // waves per centroid-tile workgroup
constexpr int kTileThreads = 64 * kTileWaves;

struct AttnArgs {
  const int32_t* assign;
  float* qc;
  const int32_t* sizes;
  const int32_t* offsets;
  const int32_t* members;
  const void* q;
  const void* k;
  const void* v;
  const int32_t* lengths;
  int heads, N, C, nchunk, topk;
  int ntile, ncg, units;  // 16-centroid tiles, 4-cluster groups, (batch, head) units
  int pchunk;             // keys per chunk of the partial states that the merge combines
  int npc;                // chunks of the partial single-pass kernel (nchunk is the state stride)
  int nsg;                // groups of four sparse_kernel work items per unit
  float scale;
  const int32_t* topk_in;
  float* pm;
  float* pz;
  float* pacc;
  int32_t* cand_idx;
  float* cand_val;
  int32_t* topk_out;
  float* mass;
  float* vcb;
  float* stats;
  void* out;
};

// MODE: 1 improved single chunk, 2 clustered partial, 3 improved partial,
// 4 oracle-top single chunk, 5 oracle-top partial (the clustered variant in
// a single chunk is attn_flash_kernel).  In the oracle-top modes the rows are the queries themselves
// (row j = query j of the unit): the top-k search is the improved one, and
// the fused mode writes each query's output from its T straight away (no
// values phase); the partial mode stops after its candidates.
//
// Row statistics come from where the data already is: while the logits of a
// key tile sit in the result registers of the first product, each lane (one
// of the 32 slices of a centroid row: eight waves x four lane groups) keeps its
// running maximum and, for the improved variant, its four largest logits.
// The row maximum is the maximum of the slice maxima; the normaliser z is the
// sum of the same exponentials that the second product uses (plus, in the
// fused improved case, those of T, which the second product leaves out); the
// top-k threshold is the k-th largest of the slices' kept values (k <= 64;
// larger k take it from a sweep of the row).
template <int D, typename T, int MODE>
__global__ __launch_bounds__(kTileThreads) void attn_tile_kernel(AttnArgs a) {
  static_assert(MODE >= 1 && MODE <= 5, "mode");
  constexpr bool OTOP = MODE >= 4;
  constexpr bool IMPROVED = (MODE & 1) != 0 || OTOP;
  constexpr bool FUSED = MODE < 2 || MODE == 4;
  constexpr int KS = D / 4, DT = D / 16;
  constexpr int NW = kTileWaves;       // waves; wave w takes key tiles w, w + NW, ...
  constexpr int NS = NW * 4;           // slices per row: (wave, lane group)
  constexpr int BT = 256 / D;          // key tiles per batch of loads (64 registers of operands)
  constexpr int NT = IMPROVED ? 4 : 1; // logits each lane keeps per row for the threshold
  __shared__ __align__(16) float logits[16 * kLStride];
  __shared__ float rowm[16], rowmass[16], rowtop[16];
  __shared__ int tcnt[16];
  __shared__ float zpart[NW][16];                              // per-wave sums of P per row
  // [row][slice] maxima and kept logits, one slice of padding per row so that
  // the slices' stores fall in distinct banks
  __shared__ float smax[16][NS + 1];
  __shared__ __align__(16) float stop[IMPROVED ? 16 : 1][NS + 1][NT];
  __shared__ uint16_t tpos16[IMPROVED ? 16 : 1][kCandCap];     // top-k candidates, then T
  __shared__ int moff[17];  // the tile's member offsets (fused modes) or sizes
  __shared__ int any_nonempty;

  // tile fastest, then chunk, then (batch, head): the tiles that read the same
  // key chunk run together on one XCD and share its L2
  const int wi = xcd_work_item();
  if (wi >= a.nchunk * a.ntile * a.units) return;
  const int tile = wi % a.ntile, chunk = (wi / a.ntile) % a.nchunk, u = wi / (a.nchunk * a.ntile);
  const int n = unit_length(a.lengths, u / a.heads, a.N);
  if constexpr (OTOP) {
    const int r0 = tile * 16;
    if (r0 >= n) {  // rows past the sequence: zero output, no top-k set (the merge
                    // writes them when there are several chunks)
      if constexpr (FUSED) {
        T* ou = static_cast<T*>(a.out) + (static_cast<size_t>(u) * a.N + r0) * D;
        for (int x = threadIdx.x; x < 16 * D; x += kTileThreads)
          if (r0 + x / D < a.C) store1(ou + x, 0.0f);
        for (int x = threadIdx.x; x < 16 * a.topk; x += kTileThreads)
          if (r0 + x / a.topk < a.C) a.topk_out[(static_cast<size_t>(u) * a.C + r0) * a.topk + x] = -1;
      }
      return;
    }
  }
  const int C = a.C;
  const int j0 = tile * 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // single-chunk improved mode: a tile whose clusters are all empty exports
  // what an empty cluster has (values 0, no top-k set, mass 0)
  auto export_empty_tile = [&]() {
    const size_t uj0 = static_cast<size_t>(u) * C + j0;
    for (int x = tid; x < 16 * D; x += kTileThreads)
      if (j0 + x / D < C) a.vcb[uj0 * D + x] = 0.0f;
    for (int x = tid; x < 16 * a.topk; x += kTileThreads)
      if (j0 + x / a.topk < C) a.topk_out[uj0 * a.topk + x] = -1;
    if (tid < 16 && j0 + tid < C) a.mass[uj0 + tid] = 0.0f;
  };
  const int k0 = chunk * kChunk;
  if (k0 >= n) {  // in a single-chunk mode: a sequence of length 0
    if constexpr (FUSED && !OTOP) export_empty_tile();
    return;
  }
  const int kn = min(kChunk, n - k0);
  const int c = lane & 15, g = lane >> 4;
  const T* ku = static_cast<const T*>(a.k) + (static_cast<size_t>(u) * a.N + k0) * D;
  const T* vu = static_cast<const T*>(a.v) + (static_cast<size_t>(u) * a.N + k0) * D;
  const int nkt = (kn + 15) / 16;
  // batches of this wave that hold tiles of the chunk (0 when it has none)
  const int nbw = (nkt - wave + NW * (BT / 2) - 1) / (NW * (BT / 2));
  // the chunk's keys and values as buffers: rows past kn read as 0
  constexpr uint32_t ESZ = sizeof(T);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(ku, static_cast<uint32_t>(kn) * D * ESZ);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vu, static_cast<uint32_t>(kn) * D * ESZ);

  // the tile's cluster sizes (or member offsets) are requested first, by
  // every thread and without a branch, so that waiting for them leaves the
  // rows of this tile and the first batch of key tiles, requested next, in
  // flight
  int pre = 0;
  if constexpr (OTOP) {
  } else if constexpr (FUSED) {
    pre = a.offsets[static_cast<size_t>(u) * (C + 1) + min(j0 + min(tid, 16), C)];
  } else {
    pre = a.sizes[static_cast<size_t>(u) * C + min(j0 + (tid & 15), C - 1)];
  }
  float bq[KS];
  if constexpr (OTOP) {  // the query rows j0 .. j0 + 15 (rows past n read as 0)
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(static_cast<const T*>(a.q) + (static_cast<size_t>(u) * a.N + j0) * D,
                  static_cast<uint32_t>(min(16, n - j0)) * D * ESZ);
    buf_load<KS>(rq, (c * D + g * KS) * ESZ, 0, bq, T{});
  } else {
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(a.qc + (static_cast<size_t>(u) * C + j0) * D, static_cast<uint32_t>(min(16, C - j0)) * D * 4);
    buf_load<KS>(rq, (c * D + g * KS) * 4, 0, bq, float{});
  }
  // key and value tiles come in batches of HB tiles (kt0, kt0 + NW, ...), two
  // batches in flight: the next one is requested before the current one is
  // used.  Every load is issued without a branch (tiles past the chunk read 0
  // through the buffer resource and cost no memory traffic), so that the
  // compiler knows how many loads are in flight and waits for the current
  // batch alone.
  constexpr int HB = BT / 2;
  static_assert(HB % 2 == 0, "tile pairs");
  // batches of a wave over a whole chunk; the loops below run as straight-line
  // code over the number of batches that hold the wave's tiles (nbw, one
  // instance per count), tiles past the chunk in the last batch computing
  // nothing
  constexpr int NB = kChunk / 16 / NW / HB;
  static_assert(NB * HB * NW * 16 == kChunk, "batches cover the chunk");
  float ka0[HB][KS], ka1[HB][KS];
  auto load_keys = [&](int kt0, float (&ka)[HB][KS]) {
    const uint32_t voff = ((kt0 * 16 + c) * D + g * KS) * ESZ;
#pragma unroll
    for (int b = 0; b < HB; ++b) buf_load<KS>(rk, voff, NW * b * 16 * D * ESZ, ka[b], T{});
  };
  load_keys(wave, ka0);

  // ---- sizes (fused: the member offsets of the 16 clusters) -----------------------
  if constexpr (OTOP) {
  } else if constexpr (FUSED) {
    if (tid < 17) moff[tid] = pre;
    __syncthreads();
    if (moff[16] == moff[0]) {  // every cluster of the tile is empty
      export_empty_tile();
      return;
    }
  } else {
    if (tid == 0) any_nonempty = 0;
    __syncthreads();
    if (tid < 16 && j0 + tid < C && pre > 0) any_nonempty = 1;
    if (tid < 16) moff[tid] = pre;  // the sizes, for the row phase
    __syncthreads();
    if (!any_nonempty) return;
  }

  // ---- logits of this chunk, with the slice statistics -------------------------------
  {
    // bf16 inputs: exact keys, the rows split into three bf16 parts, three
    // part products per 32 dims on the bf16 matrix cores (fp32-accurate
    // logits; the k index maps to the lane's own dims g KS + 8 m + j)
    constexpr bool BF = sizeof(T) == 2 || kSplitF32;
    constexpr int NC = KS / 8;
    Split8 qs[BF ? NC : 1];
    if constexpr (BF) {
#pragma unroll
      for (int m = 0; m < NC; ++m) qs[m] = split8(&bq[8 * m]);
    }
    float lmax = -INFINITY;
    float top[NT];
#pragma unroll
    for (int e = 0; e < NT; ++e) top[e] = -INFINITY;
    auto key_batch = [&](int kt0, const float (&ka)[HB][KS]) {
#pragma unroll
      for (int b = 0; b < HB; ++b) {
        const int kt = kt0 + NW * b;
        if (kt < nkt) {
          v4f acc = {0.f, 0.f, 0.f, 0.f};
          if constexpr (BF) {
#pragma unroll
            for (int m = 0; m < NC; ++m) acc = mfma_bf16x<T>(&ka[b][8 * m], qs[m], acc);
          } else {
#pragma unroll
            for (int s = 0; s < KS; ++s) acc = mfma_f32_16x16x4(ka[b][s], bq[s], acc);
          }
          float o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            o[i] = (kt * 16 + 4 * g + i < kn) ? acc[i] * a.scale : -INFINITY;
            lmax = fmaxf(lmax, o[i]);
            if constexpr (IMPROVED) {
              float v = o[i];
#pragma unroll
              for (int e = 0; e < NT; ++e) {  // insertion into the descending list
                const float hi = fmaxf(top[e], v);
                v = fminf(top[e], v);
                top[e] = hi;
              }
            }
          }
          *reinterpret_cast<float4*>(&logits[c * kLStride + kt * 16 + 4 * g]) = make_float4(o[0], o[1], o[2], o[3]);
        }
      }
    };
    // the first batch is in flight already
    with_count<NB>(nbw, [&](auto nbc) {
      constexpr int NBX = decltype(nbc)::value;
#pragma unroll
      for (int bb = 0; bb < NBX; bb += 2) {
        const int kt0 = wave + bb * NW * HB, kt1 = kt0 + NW * HB;
        if (bb + 1 < NBX) load_keys(kt1, ka1);
        key_batch(kt0, ka0);
        if (bb + 2 < NBX) load_keys(kt1 + NW * HB, ka0);
        if (bb + 1 < NBX) key_batch(kt1, ka1);
      }
    });
    // slice (wave, g) of row c
    smax[c][wave * 4 + g] = lmax;
    if constexpr (IMPROVED) {
#pragma unroll
      for (int e = 0; e < NT; e += 4)
        *reinterpret_cast<float4*>(&stop[c][wave * 4 + g][e]) = make_float4(top[e], top[e + 1], top[e + 2], top[e + 3]);
      // the top-k sweep reads each row up to 32 grp_block_len(kn): -inf past the last key tile
      const int w = 32 * grp_block_len<32>(kn) - nkt * 16;
      for (int x = tid; x < 16 * w; x += kTileThreads) logits[(x / w) * kLStride + nkt * 16 + x % w] = -INFINITY;
    }
  }
  __syncthreads();

  // ---- row maximum and top-k ----------------------------------------------------------
  // wave w owns rows 2w and 2w + 1, one 32-lane group per row, both at once;
  // lane c32 of a group reads slice c32
  static_assert(NW == 8 && NS == 32, "two rows per wave, one slice per lane");
  {
    constexpr int GL = 32;
    const int g2 = lane >> 5, c32 = lane & 31;
    const int r = wave * 2 + g2;
    const int j = j0 + r;
    float* row = &logits[r * kLStride];
    const float mx = grp_max<GL>(smax[r][c32]);
    if constexpr (IMPROVED) {
      const int kk = min(a.topk, kn);
      const size_t uj = static_cast<size_t>(u) * C + (j < C ? j : 0);
      const int jsize = OTOP ? (j < n ? 1 : 0) : j >= C ? 0 : FUSED ? moff[r + 1] - moff[r] : moff[r];
      uint16_t* cand = tpos16[r];
      int cnt;
      if (FUSED && !OTOP && a.topk_in != nullptr) {
        // caller-supplied set: its entries up to the first negative or
        // out-of-range one, in the given order
        const int32_t* tin = a.topk_in + uj * a.topk;
        int first_bad = a.topk;
        for (int x = c32; x < a.topk; x += GL) {
          const int key = tin[x];
          if ((key < 0 || key >= kn) && x < first_bad) first_bad = x;
        }
        first_bad = -static_cast<int>(grp_max<GL>(static_cast<float>(-first_bad)));
        cnt = jsize > 0 ? min(first_bad, kCandCap) : 0;
        for (int x = c32; x < cnt; x += GL) cand[x] = static_cast<uint16_t>(tin[x]);
        wave_lds_sync();
      } else {
        const int kr = jsize > 0 ? kk : 0;
        uint32_t tau;
        if (kk <= 16 * NT) {  // the slices' lists: 32 * NT values per row, at least 2 kk
          uint32_t keys[NT];
#pragma unroll
          for (int e = 0; e < NT; ++e) {
            const float v = stop[r][c32][e];
            keys[e] = v > -INFINITY ? order_key(v) : 0u;
          }
          tau = group_kth_key<NT, GL>(keys, kr);
        } else {  // a sweep of the row: 8 values per lane, 256 per row, at least 2 kk
          tau = group_row_threshold<8, GL>(row, kn, kr);
        }
        cnt = group_select<kCandCap, GL>(row, kn, kr, tau, cand);
        // rows whose threshold let too many entries through (many ties): the
        // whole wave selects them one after the other; its scratch is the
        // slice area of its own two rows, consumed by now
        static_assert(!IMPROVED || 2 * (NS + 1) * NT >= 2 * kCandCap, "two rows' slices hold the wave's scratch");
        const uint64_t over = __ballot(cnt < 0);
        for (int gg = 0; gg < 2; ++gg) {
          if (((over >> (32 * gg)) & 1ull) == 0ull) continue;
          const int rg = wave * 2 + gg;
          float md, zd;
          const int cg = wave_topk_row<kCandCap>(&logits[rg * kLStride], kn, kk,
                                                 reinterpret_cast<int*>(&stop[2 * wave][0][0]),
                                                 tpos16[rg], &md, &zd);
          wave_lds_sync();
          if (g2 == gg) cnt = cg;
        }
      }
      // sum over T of exp(s - max) (the numerator of the mass; a chunk of
      // several leaves it to the merge)
      float tsum = 0.0f;
      if constexpr (FUSED) {
        for (int x = c32; x < cnt; x += GL) tsum += __expf(row[cand[x]] - mx);
        tsum = grp_sum<GL>(tsum);
      }
      if constexpr (OTOP && FUSED) {
        // out_j = sum_{l in T} exp(s_l - m) v_l / sum_{l in T} exp(s_l - m), the
        // row maximum m being in T; lane c32 takes dims c32 (and c32 + 32),
        // eight value rows in flight
        constexpr int DPL = D / GL;
        const T* vrow = static_cast<const T*>(a.v) + static_cast<size_t>(u) * a.N * D;
        float o[DPL];
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[e] = 0.0f;
        for (int x0 = 0; x0 < cnt; x0 += 8) {
          int pos[8];
          float pv[8], vv[8][DPL];
#pragma unroll
          for (int e = 0; e < 8; ++e) pos[e] = x0 + e < cnt ? cand[x0 + e] : -1;
#pragma unroll
          for (int e = 0; e < 8; ++e)
#pragma unroll
            for (int f = 0; f < DPL; ++f)
              vv[e][f] = pos[e] >= 0 ? to_f32(vrow[static_cast<size_t>(pos[e]) * D + c32 + GL * f]) : 0.0f;
#pragma unroll
          for (int e = 0; e < 8; ++e) pv[e] = pos[e] >= 0 ? __expf(row[pos[e]] - mx) : 0.0f;
#pragma unroll
          for (int e = 0; e < 8; ++e)
#pragma unroll
            for (int f = 0; f < DPL; ++f) o[f] = fmaf(pv[e], vv[e][f], o[f]);
        }
        const float inv = cnt > 0 ? 1.0f / tsum : 0.0f;
        if (j < C) {
          T* orow = static_cast<T*>(a.out) + (static_cast<size_t>(u) * a.N + j) * D;
#pragma unroll
          for (int f = 0; f < DPL; ++f) store1(orow + c32 + GL * f, o[f] * inv);
          for (int x = c32; x < a.topk; x += GL) a.topk_out[uj * a.topk + x] = x < cnt ? cand[x] : -1;
        }
      } else if constexpr (FUSED) {
        // T masked out of the row so that P V gives the rest part
        wave_lds_sync();
        for (int x = c32; x < cnt; x += GL) row[cand[x]] = -INFINITY;
        if (j < C)
          for (int x = c32; x < a.topk; x += GL) a.topk_out[uj * a.topk + x] = x < cnt ? cand[x] : -1;
        if (c32 == 0) tcnt[r] = cnt;
      } else {
        if (j < C) {
          const size_t cb = (uj * a.nchunk + chunk) * a.topk;
          for (int x = c32; x < a.topk; x += GL) {
            const bool ok = x < cnt;
            const int pos = ok ? cand[x] : 0;
            a.cand_idx[cb + x] = ok ? k0 + pos : -1;
            a.cand_val[cb + x] = ok ? row[pos] : -INFINITY;
          }
        }
      }
      if (c32 == 0) rowtop[r] = tsum;
      wave_lds_sync();
    }
    if (c32 == 0) rowm[r] = mx;
  }
  if constexpr (OTOP) return;  // outputs written, or candidates for the merge
  __syncthreads();

  // ---- values: O^T = V^T P^T (P = exp(S - m), T masked in the fused improved case)
  v4f oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = v4f{0.f, 0.f, 0.f, 0.f};
  float psum = 0.0f;
  {
    const float mc = rowm[c];
    float va0[HB][4][DT], va1[HB][4][DT];
    auto load_vals = [&](int kt0, float (&va)[HB][4][DT]) {
      const uint32_t voff = ((kt0 * 16 + 4 * g) * D + DT * c) * ESZ;
#pragma unroll
      for (int b = 0; b < HB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) buf_load<DT>(rv, voff, (NW * b * 16 + i) * D * ESZ, va[b][i], T{});
    };
    auto value_batch = [&](int kt0, const float (&va)[HB][4][DT]) {
      if constexpr (sizeof(T) == 2 || kSplitF32) {
        // bf16 values are exact and P keeps two bf16 parts (mfma_weights);
        // tiles b and b + 1 of the batch form one product over 32 keys (k = 8 g + j: key
        // 4 g + j of tile b for j < 4, of tile b + 1 otherwise), a tile past
        // the row contributing P = 0
#pragma unroll
        for (int b = 0; b < HB; b += 2) {
          if (kt0 + NW * b >= nkt) break;
          float p8[8];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int kt = kt0 + NW * (b + h);
            if (kt < nkt) {
              const float4 s4 = *reinterpret_cast<const float4*>(&logits[c * kLStride + kt * 16 + 4 * g]);
              p8[4 * h] = __expf(s4.x - mc);
              p8[4 * h + 1] = __expf(s4.y - mc);
              p8[4 * h + 2] = __expf(s4.z - mc);
              p8[4 * h + 3] = __expf(s4.w - mc);
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i) p8[4 * h + i] = 0.0f;
            }
          }
          psum += ((p8[0] + p8[1]) + (p8[2] + p8[3])) + ((p8[4] + p8[5]) + (p8[6] + p8[7]));
          const Split8 ps = split8(p8);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            float v8[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              v8[i] = va[b][i][dt];
              v8[4 + i] = va[b + 1][i][dt];
            }
            oacc[dt] = mfma_weights<T>(v8, ps, oacc[dt]);
          }
        }
      } else {
#pragma unroll
        for (int b = 0; b < HB; ++b) {
          const int kt = kt0 + NW * b;
          if (kt < nkt) {
            const float4 s4 = *reinterpret_cast<const float4*>(&logits[c * kLStride + kt * 16 + 4 * g]);
            const float p[4] = {__expf(s4.x - mc), __expf(s4.y - mc), __expf(s4.z - mc), __expf(s4.w - mc)};
            psum += (p[0] + p[1]) + (p[2] + p[3]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
              for (int dt = 0; dt < DT; ++dt) oacc[dt] = mfma_f32_16x16x4(va[b][i][dt], p[i], oacc[dt]);
          }
        }
      }
    };
    with_count<NB>(nbw, [&](auto nbc) {
      constexpr int NBX = decltype(nbc)::value;
      load_vals(wave, va0);
#pragma unroll
      for (int bb = 0; bb < NBX; bb += 2) {
        const int kt0 = wave + bb * NW * HB, kt1 = kt0 + NW * HB;
        if (bb + 1 < NBX) load_vals(kt1, va1);
        value_batch(kt0, va0);
        if (bb + 2 < NBX) load_vals(kt1 + NW * HB, va0);
        if (bb + 1 < NBX) value_batch(kt1, va1);
      }
    });
  }
  psum = cross_rows_sum(psum);
  if (g == 0) zpart[wave][c] = psum;
  __syncthreads();  // logits are dead from here on: reuse them
  // [NW waves][16 centroids][D + kRedPad]: each lane stores its DT
  // consecutive dimensions of a row at once, the padded rows in distinct banks
  constexpr int RS = D + kRedPad;
  float* red = logits;
  static_assert(NW * 16 * RS <= 16 * kLStride, "logit area reuse");
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float* dst = &red[(wave * 16 + c) * RS + DT * (4 * g + i)];
    if constexpr (DT == 4)
      *reinterpret_cast<float4*>(dst) = make_float4(oacc[0][i], oacc[1][i], oacc[2][i], oacc[3][i]);
    else
      *reinterpret_cast<float2*>(dst) = make_float2(oacc[0][i], oacc[1][i]);
  }
  __syncthreads();
  for (int x = tid; x < 16 * D; x += kTileThreads) {
    const int cc = x / D, dim = x % D;
    float sum = 0.0f, z = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      sum += red[(w * 16 + cc) * RS + dim];
      z += zpart[w][cc];
    }
    if constexpr (IMPROVED && FUSED) z += rowtop[cc];
    if (j0 + cc >= C) continue;
    const size_t ujc = static_cast<size_t>(u) * C + j0 + cc;
    if constexpr (FUSED) {
      const bool nonempty = moff[cc + 1] > moff[cc];
      const float val = nonempty ? sum / z : 0.0f;
      a.vcb[ujc * D + dim] = val;
      if (dim == 0) {  // softmax statistics for the backward pass
        a.stats[ujc * 2] = rowm[cc];
        a.stats[ujc * 2 + 1] = z;
      }
      if (IMPROVED && dim == 0) {
        const float mass = nonempty ? rowtop[cc] / z : 0.0f;
        rowmass[cc] = mass;
        a.mass[ujc] = mass;
      }
    } else {
      const size_t pj = ujc * a.nchunk + chunk;
      a.pacc[pj * D + dim] = sum;
      if (dim == 0) {
        a.pm[pj] = rowm[cc];
        a.pz[pj] = z;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Clustered centroid attention over one key chunk in a single pass (Eqs. 4-6):
// the centroid logits never leave the registers.  Wave w takes key tiles
// w, w + kFlashWaves, ...; for each tile the logits S^T = K Q^c^T come from
// the fp32 matrix cores in the layout that the second product wants for P^T,
// so each lane keeps, for its centroid column, a running maximum m, the sum z
// of exp(s - m) over its keys and the partial O^T = V^T P^T, both rescaled by
// exp(m_old - m_new) when the maximum grows.  The waves' (m, z, O) are merged
// in LDS (log-sum-exp), which gives V^c_j and the softmax statistics; then
// every member row receives V^c_j (Eq. 6).
//
// PARTIAL: the same pass over one chunk of a.pchunk keys per workgroup
// (several chunks of a long sequence), writing the chunk's (m, z,
// unnormalised values) for attn_merge_kernel instead of the member rows.
// ---------------------------------------------------------------------------
constexpr int kFlashWaves = 8;
constexpr int kFlashThreads = 64 * kFlashWaves;
// keys per workgroup of the partial pass: kFlashChunk, or twice that when
// the grid still fills most of the chip (flash_chunk)
constexpr int kFlashChunk = 2048;
static_assert(kFlashChunk % kChunk == 0, "partial states at the stride of kChunk chunks");

template <int D, typename T, bool PARTIAL>
__global__ __launch_bounds__(kFlashThreads) void attn_flash_kernel(AttnArgs a) {
  constexpr int KS = D / 4, DT = D / 16, NW = kFlashWaves;
  constexpr uint32_t ESZ = sizeof(T);
  __shared__ float red[NW][16][D + 1];  // per-wave O^T partials, [wave][centroid][dim]
  __shared__ float wm[NW][16], wz[NW][16];
  __shared__ __align__(16) float vhat[16][D];
  __shared__ int moff[17];
  __shared__ int mlist[PARTIAL ? 1 : kChunk];

  // tile fastest, (then chunk,) then (batch, head): the tiles that read the
  // same keys run together on one XCD and share its L2
  const int wi = xcd_work_item();
  const int nfc = PARTIAL ? a.npc : 1;
  if (wi >= nfc * a.ntile * a.units) return;
  const int tile = wi % a.ntile, chunk = (wi / a.ntile) % nfc, u = wi / (nfc * a.ntile);
  const int nu = unit_length(a.lengths, u / a.heads, a.N);
  const int k0 = PARTIAL ? chunk * a.pchunk : 0;
  if (PARTIAL && k0 >= nu) return;  // a chunk past the sequence: the merge does not read it
  const int n = PARTIAL ? min(a.pchunk, nu - k0) : nu;  // keys of this workgroup
  const int C = a.C;
  const int j0 = tile * 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, g = lane >> 4;
  // the centroid rows and (fp32) the first key tile do not depend on the
  // member offsets: they are requested first, so that both latencies overlap
  const T* ku = static_cast<const T*>(a.k) + (static_cast<size_t>(u) * a.N + k0) * D;
  const T* vu = static_cast<const T*>(a.v) + (static_cast<size_t>(u) * a.N + k0) * D;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(ku, static_cast<uint32_t>(n) * D * ESZ);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vu, static_cast<uint32_t>(n) * D * ESZ);
  const int nkt = (n + 15) / 16;
  float bq[KS];
  {
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(a.qc + (static_cast<size_t>(u) * C + j0) * D, static_cast<uint32_t>(min(16, C - j0)) * D * 4);
    buf_load<KS>(rq, (c * D + g * KS) * 4, 0, bq, float{});
  }
  // fp32 inputs: one key tile in registers, the next one requested before
  // the current one goes to the fp32 matrix cores (two buffers used in turn)
  float kbuf[2][KS], vbuf[2][4][DT];
  auto load_tile = [&](int kt, float* kx, float (*vx)[DT]) {
    buf_load<KS>(rk, ((kt * 16 + c) * D + g * KS) * ESZ, 0, kx, T{});
    const uint32_t voff = ((kt * 16 + 4 * g) * D + DT * c) * ESZ;
#pragma unroll
    for (int i = 0; i < 4; ++i) buf_load<DT>(rv, voff, i * D * ESZ, vx[i], T{});
  };
  if constexpr (sizeof(T) == 4 && !kSplitF32) load_tile(wave, kbuf[0], vbuf[0]);
  const int32_t* ou = a.offsets + static_cast<size_t>(u) * (C + 1);
  if (tid < 17) moff[tid] = ou[min(j0 + tid, C)];
  __syncthreads();
  if (moff[16] == moff[0] || n == 0) {  // every cluster of the tile is empty: V^c = 0
    if constexpr (PARTIAL) return;       // (the merge writes it)
    const size_t uj0 = static_cast<size_t>(u) * C + j0;
    for (int x = tid; x < 16 * D; x += kFlashThreads)
      if (j0 + x / D < C) a.vcb[uj0 * D + x] = 0.0f;
    return;
  }
  const int m0 = moff[0], mn = moff[16] - m0;
  // the member lists are requested now and stored once the products are done
  constexpr int MPT = PARTIAL ? 1 : kChunk / kFlashThreads;
  int mreg[MPT];
  if constexpr (!PARTIAL) {
    const int32_t* mg = a.members + static_cast<size_t>(u) * a.N + m0;
#pragma unroll
    for (int e = 0; e < MPT; ++e) {
      const int x = tid + kFlashThreads * e;
      mreg[e] = x < mn ? mg[x] : 0;
    }
  }
  float mrun = -INFINITY, zl = 0.0f;
  v4f oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = v4f{0.f, 0.f, 0.f, 0.f};
  if constexpr (sizeof(T) == 2 || kSplitF32) {
    // Both products on the bf16 matrix cores.  Q^c is split into three bf16
    // parts (an fp32 value is exactly the sum of its three truncated parts), so
    // that every logit keeps fp32 accuracy: bf16 keys are exact (three part
    // products per 32 dims); P keeps two parts against the exact bf16 values
    // (mfma_weights, each weight short by under 2^-15 of itself); fp32 keys
    // and values are split too (six part products, mfma_split6).  The k
    // index of a product over dims maps to the lane's own dims g KS + 8 m + j;
    // over keys, k = 8 g + j is key 4 g + j of the block's first tile (j < 4)
    // or key 4 g + j - 4 of its second, which is where the logit results put
    // P.
    constexpr int NC = KS / 8;              // 32-dim chunks
    Split8 qs[NC];
#pragma unroll
    for (int m = 0; m < NC; ++m) qs[m] = split8(&bq[8 * m]);
    const int nkb = (n + 31) / 32;  // blocks of two key tiles; wave w takes blocks w, w + NW, ...
    // every load is issued, rows past n reading as 0, so that the compiler
    // counts them and each block waits only for its own rows
    auto load_block = [&](int bk, float (*kx)[KS], float (*vx)[4][DT]) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int kt = 2 * bk + t;
        buf_load<KS>(rk, ((kt * 16 + c) * D + g * KS) * ESZ, 0, kx[t], T{});
        const uint32_t voff = ((kt * 16 + 4 * g) * D + DT * c) * ESZ;
#pragma unroll
        for (int i = 0; i < 4; ++i) buf_load<DT>(rv, voff, i * D * ESZ, vx[t][i], T{});
      }
    };
    auto step = [&](int bk, float (*kx)[KS], float (*vx)[4][DT]) {
      float o[8];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < NC; ++m) {
          acc = mfma_bf16x<T>(&kx[t][8 * m], qs[m], acc);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) o[4 * t + i] = ((2 * bk + t) * 16 + 4 * g + i < n) ? acc[i] * a.scale : -INFINITY;
      }
      // key 32 bk is valid, so the block maximum of every column is finite
      float bmax = o[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) bmax = fmaxf(bmax, o[e]);
      const float mnew = fmaxf(mrun, cross_rows_max(bmax));
      const float alpha = __expf(mrun - mnew);  // 0 on the first block
      mrun = mnew;
      float p[8], psum = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = __expf(o[e] - mnew);
        psum += p[e];
      }
      zl = zl * alpha + psum;
      const Split8 ps = split8(p);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        float va8[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          va8[j] = vx[0][j][dt];
          va8[4 + j] = vx[1][j][dt];
        }
        oacc[dt] = mfma_weights<T>(va8, ps, oacc[dt] * alpha);
      }
    };
    for (int bk = wave; bk < nkb; bk += NW) {
      float kx[2][KS], vx[2][4][DT];
      load_block(bk, kx, vx);
      step(bk, kx, vx);
    }
  } else {
    // fp32 inputs on the fp32 matrix cores (kSplitF32 false): the loop is
    // unrolled so that no buffer is copied; every
    // load is issued, rows past n reading as 0, so that the compiler counts
    // them and each tile waits only for its own rows (the first tile was
    // requested before the offsets)
    auto step = [&](int kt, const float* kx, const float (*vx)[DT]) {
      v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) acc = mfma_f32_16x16x4(kx[s], bq[s], acc);
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = (kt * 16 + 4 * g + i < n) ? acc[i] * a.scale : -INFINITY;
      // key kt * 16 is valid, so the tile maximum of every column is finite
      const float tmax = cross_rows_max(fmaxf(fmaxf(o[0], o[1]), fmaxf(o[2], o[3])));
      const float mnew = fmaxf(mrun, tmax);
      const float alpha = __expf(mrun - mnew);  // 0 on the first tile
      mrun = mnew;
      float p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) p[i] = __expf(o[i] - mnew);
      zl = zl * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 4; ++r) oacc[dt][r] *= alpha;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[dt] = mfma_f32_16x16x4(vx[i][dt], p[i], oacc[dt]);
    };
    for (int kt0 = wave; kt0 < nkt; kt0 += 2 * NW) {
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int kt = kt0 + NW * e;
        // the buffer of the next tile is the one that the previous step freed
        load_tile(kt + NW, kbuf[(e + 1) % 2], vbuf[(e + 1) % 2]);
        if (kt < nkt) step(kt, kbuf[e], vbuf[e]);
      }
    }
  }
  const float zc = cross_rows_sum(zl);
  if (g == 0) {
    wm[wave][c] = mrun;
    wz[wave][c] = zc;
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) red[wave][c][DT * (4 * g + r) + dt] = oacc[dt][r];
  if constexpr (!PARTIAL) {
#pragma unroll
    for (int e = 0; e < MPT; ++e) {
      const int x = tid + kFlashThreads * e;
      if (x < mn) mlist[x] = mreg[e];
    }
  }
  __syncthreads();
  for (int x = tid; x < 16 * D; x += kFlashThreads) {
    const int cc = x / D, dim = x % D;
    float M = wm[0][cc];
#pragma unroll
    for (int w = 1; w < NW; ++w) M = fmaxf(M, wm[w][cc]);
    float Z = 0.0f, O = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float f = __expf(wm[w][cc] - M);  // 0 for a wave without keys
      Z += f * wz[w][cc];
      O += f * red[w][cc][dim];
    }
    if (j0 + cc >= C) continue;
    const size_t ujc = static_cast<size_t>(u) * C + j0 + cc;
    if constexpr (PARTIAL) {  // the chunk's state, relative to its maximum M
      const size_t pj = ujc * a.nchunk + chunk;
      a.pacc[pj * D + dim] = O;
      if (dim == 0) {
        a.pm[pj] = M;
        a.pz[pj] = Z;
      }
      continue;
    }
    const bool nonempty = moff[cc + 1] > moff[cc];
    const float val = nonempty ? O / Z : 0.0f;
    vhat[cc][dim] = val;
    a.vcb[ujc * D + dim] = val;
    if (dim == 0) {  // softmax statistics for the backward pass
      a.stats[ujc * 2] = M;
      a.stats[ujc * 2 + 1] = Z;
    }
  }
  if constexpr (PARTIAL) return;
  __syncthreads();
  // Eq. (6): each member row receives V^c_j; a lane writes 4 dims of a row
  T* out = static_cast<T*>(a.out) + static_cast<size_t>(u) * a.N * D;
  constexpr int RPW = 16 / NW;  // clusters per wave
  constexpr int LPR = D / 4, RPS = 64 / LPR;
  const int part = lane % LPR, sub = lane / LPR;
  for (int rr = 0; rr < RPW; ++rr) {
    const int r = wave * RPW + rr;
    if (j0 + r >= C) break;
    const int sz = moff[r + 1] - moff[r];
    const int* mem = mlist + (moff[r] - m0);
    const float4 val = *reinterpret_cast<const float4*>(&vhat[r][part * 4]);
    for (int m1 = sub; m1 < sz; m1 += RPS) {
      const int qrow = mem[m1];
      store4(out + static_cast<size_t>(qrow) * D + part * 4, val.x, val.y, val.z, val.w);
    }
  }
}

// ---------------------------------------------------------------------------
// Merge of the chunks (several chunks only).  OTOP (oracle-top, IMPROVED
// set): row j is query j; its T comes from the chunks' candidates as in the
// improved case, and the output row is the softmax over T of the candidates'
// logits applied to the T rows of V.
// ---------------------------------------------------------------------------
template <int D, typename T, bool IMPROVED, bool OTOP = false>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  __shared__ int cscr[4][2 * kCandCap];  // per-wave top-k scratch
  __shared__ int selout[4][128];
  __shared__ float selval[4][128];
  __shared__ float vcs[4][D];
  const int wi = xcd_work_item();  // cluster group fastest, then (batch, head)
  if (wi >= a.ncg * a.units) return;
  const int u = wi / a.ncg, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int C = a.C;
  const int j = (wi % a.ncg) * 4 + wave;
  if (j >= C) return;
  const size_t uj = static_cast<size_t>(u) * C + j;
  const int n = unit_length(a.lengths, u / a.heads, a.N);
  const int sz = OTOP ? (j < n ? 1 : 0) : a.sizes[uj];
  if (sz == 0) {
    if constexpr (OTOP) {  // padded row
      T* orow = static_cast<T*>(a.out) + (static_cast<size_t>(u) * a.N + j) * D;
      for (int x = lane; x < D; x += 64) store1(orow + x, 0.0f);
    } else {
      for (int x = lane; x < D; x += 64) a.vcb[uj * D + x] = 0.0f;
    }
    if (IMPROVED) {
      for (int x = lane; x < a.topk; x += 64) a.topk_out[uj * a.topk + x] = -1;
      if (!OTOP && lane == 0) a.mass[uj] = 0.0f;
    }
    return;
  }
  const int nch = (n + a.pchunk - 1) / a.pchunk;
  constexpr int RPS = 64 / D;
  const int t = lane % D, r = lane / D;
  float M = -INFINITY, Z = 0.0f;
  if constexpr (!OTOP) {
    const float* pmj = a.pm + uj * a.nchunk;
    const float* pzj = a.pz + uj * a.nchunk;
    for (int x = lane; x < nch; x += 64) M = fmaxf(M, pmj[x]);
    M = wave_max(M);
    for (int x = lane; x < nch; x += 64) Z += pzj[x] * __expf(pmj[x] - M);
    Z = wave_sum(Z);
    if (lane == 0) {  // softmax statistics for the backward pass
      a.stats[uj * 2] = M;
      a.stats[uj * 2 + 1] = Z;
    }
    // V^c = sum_chunks exp(m_c - M) acc_c / Z   (lane -> dimension; eight
    // chunks' partials in flight)
    float acc = 0.0f;
#pragma unroll 8
    for (int x = r; x < nch; x += RPS) acc += __expf(pmj[x] - M) * a.pacc[(uj * a.nchunk + x) * D + t];
    if (RPS == 2) acc += lane_xor32(acc);
    const float vc = acc / Z;
    if (!IMPROVED) {
      if (lane < D) a.vcb[uj * D + t] = vc;
      return;
    }
    if (lane < D) vcs[wave][t] = vc;
  }
  const int kk = min(a.topk, n);
  const T* ku = static_cast<const T*>(a.k) + static_cast<size_t>(u) * a.N * D;
  const T* vu = static_cast<const T*>(a.v) + static_cast<size_t>(u) * a.N * D;
  int cnt;
  if (!OTOP && a.topk_in != nullptr) {
    // caller-supplied set: entries until the first negative or out-of-range one;
    // their logits are recomputed
    const int32_t* tin = a.topk_in + uj * a.topk;
    const float* qj = a.qc + uj * D;
    cnt = 0;
    while (cnt < a.topk && tin[cnt] >= 0 && tin[cnt] < n) ++cnt;
    for (int x = lane; x < cnt; x += 64) {
      const int key = tin[x];
      float dot = 0.0f;
      for (int d = 0; d < D; ++d) dot = fmaf(qj[d], to_f32(ku[static_cast<size_t>(key) * D + d]), dot);
      selout[wave][x] = key;
      selval[wave][x] = dot * a.scale;
    }
  } else {
    const int32_t* ci = a.cand_idx + uj * a.nchunk * a.topk;
    const float* cv = a.cand_val + uj * a.nchunk * a.topk;
    float mdummy, zdummy;
    cnt = wave_topk_row<kCandCap>(cv, nch * a.topk, kk, cscr[wave], selout[wave], &mdummy,
                                  &zdummy);
    wave_lds_sync();
    for (int x = lane; x < cnt; x += 64) {
      const int pos = selout[wave][x];
      selval[wave][x] = cv[pos];
      selout[wave][x] = ci[pos];
    }
  }
  wave_lds_sync();
  if constexpr (OTOP) {  // softmax over T alone
    for (int x = lane; x < cnt; x += 64) M = fmaxf(M, selval[wave][x]);
    M = wave_max(M);
    for (int x = lane; x < cnt; x += 64) Z += __expf(selval[wave][x] - M);
    Z = wave_sum(Z);
  }
  // m_j and the top-k part of A^c V (eight value rows in flight per lane group)
  float msum = 0.0f;
  for (int x = lane; x < cnt; x += 64) msum += __expf(selval[wave][x] - M) / Z;
  msum = wave_sum(msum);
  float top = 0.0f;
  int x = r;
  for (; x + 7 * RPS < cnt; x += 8 * RPS) {
    float wv[8], vv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      wv[e] = __expf(selval[wave][x + e * RPS] - M) / Z;
      vv[e] = to_f32(vu[static_cast<size_t>(selout[wave][x + e * RPS]) * D + t]);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) top += wv[e] * vv[e];
  }
  for (; x < cnt; x += RPS)
    top += (__expf(selval[wave][x] - M) / Z) * to_f32(vu[static_cast<size_t>(selout[wave][x]) * D + t]);
  if (RPS == 2) top += lane_xor32(top);
  for (int y = lane; y < a.topk; y += 64) a.topk_out[uj * a.topk + y] = y < cnt ? selout[wave][y] : -1;
  if constexpr (OTOP) {
    if (lane < D) store1(static_cast<T*>(a.out) + (static_cast<size_t>(u) * a.N + j) * D + t, top);
    return;
  }
  if (lane < D) a.vcb[uj * D + t] = vcs[wave][t] - top;
  if (lane == 0) a.mass[uj] = msum;
}

// ---------------------------------------------------------------------------
// Improved values (Section 3.3 with the supplementary decomposition), one
// wave per (cluster j, chunk of up to kSparseChunk members), so that large
// clusters spread over many waves: for every member i,
//   out_i = m_j * sum_{l in T} softmax_T(q_i k_l / sqrt d)_l v_l + V^b_j.
// The loads come in three dependent steps: size, offset, m_j, V^b_j and T;
// then the member indices with the K_T and V_T rows; then the member rows of
// Q.  Member tiles after the first are requested one tile ahead.
//   S^T = K_T Q^T : A = K_T rows (slot kt*16 + lane%16, dims g*KS..), B = Q^T
//   O^T = V_T^T P^T: A = V_T^T (dims DT*(lane%16)+dt, slot kt*16+4g+i),
//                     B = P^T straight from the S^T result registers.
// Lane (query c, group g) ends with dims DT*4g .. DT*4g + 4*DT - 1 of its row.
// ---------------------------------------------------------------------------
// Register budgets that fit without spills and measured faster than the
// unconstrained allocation: seven waves per SIMD for d = 32 with k <= 32 (69
// registers in fp32, against six waves), five for bf16 d = 64 with k <= 32
// (the next member tile's rows take registers of their own)
template <int D, typename T, int NKT>
constexpr int kSparseMinWaves = (D == 32 && NKT <= 2) ? 7 : (D == 64 && NKT == 2 && sizeof(T) == 2) ? 5 : 1;
// d = 64: the next member tile's query rows are requested before the current
// tile goes through the products (d = 32 measured faster with the seven waves
// per SIMD that the registers of a second tile would cost)
template <int D>
constexpr bool kSparsePrefetch = D == 64;
template <int D, typename T, int NKT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kSparseMinWaves<D, T, NKT>))) void sparse_kernel(AttnArgs a) {
  constexpr int KS = D / 4, DT = D / 16;
  constexpr uint32_t ESZ = sizeof(T);
  constexpr uint32_t kNone = 0x80000000u;  // past every buffer: loads read 0, stores are dropped
  __shared__ int tp[4][kCandCap];
  __shared__ __align__(16) float vbs[4][D];  // V^b_j of each wave's cluster
  const int wi = xcd_work_item();  // item group fastest, then (batch, head)
  if (wi >= a.nsg * a.units) return;
  const int u = wi / a.nsg, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int C = a.C;
  // Work item t of the unit: for t < C the first kSparseChunk members of
  // cluster t; for t >= C the further chunks of the clusters that have more,
  // in cluster order (located by a prefix sum over the clusters).
  const int t = (wi % a.nsg) * 4 + wave;
  int j = t, chunk = 0;
  if (t >= C) {
    const int32_t* su = a.sizes + static_cast<size_t>(u) * C;
    const int want = t - C;
    // every cluster size requested at once (the interface admits C <= 256:
    // four per lane)
    constexpr int SPL = 256 / 64;
    int sv[SPL];
#pragma unroll
    for (int e = 0; e < SPL; ++e) sv[e] = su[min(64 * e + lane, C - 1)];
    int run = 0;
    j = -1;
#pragma unroll
    for (int e = 0; e < SPL; ++e) {
      const int x0 = 64 * e;
      if (x0 >= C) break;
      const int x = x0 + lane;
      const int s = x < C ? sv[e] : 0;
      const int extra = s > kSparseChunk ? (s - 1) / kSparseChunk : 0;
      const int incl = wave_incl_scan(extra);
      const uint64_t hit = __ballot(want >= run + incl - extra && want < run + incl);
      if (hit != 0ull) {
        const int src = __ffsll(static_cast<unsigned long long>(hit)) - 1;
        j = x0 + src;
        chunk = 1 + want - (run + __builtin_amdgcn_readlane(incl - extra, src));
        break;
      }
      run += __builtin_amdgcn_readlane(incl, 63);
    }
    if (j < 0) return;  // past the unit's last chunk
  }
  if (j >= C) return;
  const size_t uj = static_cast<size_t>(u) * C + j;

  // ---- load step 1: the cluster's size, offset, m_j, V^b_j and T ------------------
  const int sz_all = a.sizes[uj];
  const int sz = min(kSparseChunk, sz_all - chunk * kSparseChunk);  // members of this item
  const int off = a.offsets[static_cast<size_t>(u) * (C + 1) + j] + chunk * kSparseChunk;
  const float mh = a.mass[uj];
  int tv[kCandCap / 64];
#pragma unroll
  for (int e = 0; e < kCandCap / 64; ++e) {
    const int x = lane + 64 * e;
    tv[e] = x < a.topk ? a.topk_out[uj * a.topk + x] : -1;
  }
  // V^b_j is the same for every member row: it waits in LDS, not in registers
  float vb4[4];
  if (lane < D / 4) load_row<4>(a.vcb + uj * D + 4 * lane, vb4);
  if (sz <= 0) return;
  if (lane < D / 4) *reinterpret_cast<float4*>(&vbs[wave][4 * lane]) = make_float4(vb4[0], vb4[1], vb4[2], vb4[3]);
  // T: the leading non-negative entries (a caller-supplied set may be shorter)
  int kk = 0;
#pragma unroll
  for (int e = 0; e < kCandCap / 64; ++e) {
    if (tv[e] >= 0) tp[wave][lane + 64 * e] = tv[e];
    kk += __popcll(__ballot(tv[e] >= 0));
  }
  wave_lds_sync();
  const int nkt = (kk + 15) >> 4;

  // ---- load step 2: member indices of the first two tiles, K_T and V_T --------------
  const int32_t* mem = a.members + static_cast<size_t>(u) * a.N + off;
  int row0 = c < sz ? mem[c] : -1;
  int row1 = 16 + c < sz ? mem[16 + c] : -1;
  const size_t base = static_cast<size_t>(u) * a.N * D;
  const uint32_t ubytes = static_cast<uint32_t>(a.N) * D * ESZ;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(static_cast<const T*>(a.q) + base, ubytes);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(static_cast<const T*>(a.k) + base, ubytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(static_cast<const T*>(a.v) + base, ubytes);
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(static_cast<T*>(a.out) + base, ubytes);
  float kf[NKT][KS];     // K_T: slot kt * 16 + lane % 16, dims (lane / 16) * KS ..
  float vf[NKT][4][DT];  // V_T^T: slot kt * 16 + 4 (lane / 16) + i, dims (lane % 16) * DT ..
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt) {
    if (kt < nkt) {
      const int slot = kt * 16 + c;
      buf_load<KS>(rk, slot < kk ? static_cast<uint32_t>(tp[wave][slot]) * D * ESZ + g * KS * ESZ : kNone, 0,
                   kf[kt], T{});
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int sl = kt * 16 + 4 * g + i;
        buf_load<DT>(rv, sl < kk ? static_cast<uint32_t>(tp[wave][sl]) * D * ESZ + DT * c * ESZ : kNone, 0,
                     vf[kt][i], T{});
      }
    } else {
#pragma unroll
      for (int s = 0; s < KS; ++s) kf[kt][s] = 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) vf[kt][i][dt] = 0.0f;
    }
  }
  auto qoff = [&](int row) { return row >= 0 ? static_cast<uint32_t>(row) * D * ESZ + g * KS * ESZ : kNone; };

  // ---- load step 3: member rows of Q, one tile of 16 at a time --------------------
  // The member indices two tiles ahead are requested first and (d = 64) the
  // next tile's rows before the current tile goes through the products; every
  // load is issued without a branch (past the item's members they read 0
  // through their buffer resources), so that each waits for itself alone.
  const __amdgpu_buffer_rsrc_t rm = make_rsrc(mem, static_cast<uint32_t>(sz) * 4);
  constexpr bool PF = kSparsePrefetch<D>;
  float bq[KS];
  if constexpr (PF) buf_load<KS>(rq, qoff(row0), 0, bq, T{});
  for (int mt = 0; mt < sz; mt += 16) {
    const bool more = mt + 16 < sz;
    float bqn[PF ? KS : 1];
    if constexpr (PF)
      buf_load<KS>(rq, qoff(more ? row1 : -1), 0, bqn, T{});
    else
      buf_load<KS>(rq, qoff(row0), 0, bq, T{});
    const int m2 = mt + 32 + c;
    const int r2 = static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(rm, static_cast<uint32_t>(m2) * 4, 0, 0));
    const int row2 = m2 < sz ? r2 : -1;
    v4f sacc[NKT];
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
      sacc[kt] = v4f{0.f, 0.f, 0.f, 0.f};
      if (kt < nkt) {
        if constexpr (sizeof(T) == 2) {
          // bf16 inputs: the T rows of K and the member rows of Q are exact
          // bf16, so one bf16 product per 32 dims gives the fp32-accurate logits
#pragma unroll
          for (int m = 0; m < KS / 8; ++m)
            sacc[kt] = mfma_bf16_16x16x32(pack_bf16x8(&kf[kt][8 * m]), pack_bf16x8(&bq[8 * m]), sacc[kt]);
        } else {
#pragma unroll
          for (int s = 0; s < KS; ++s) sacc[kt] = mfma_f32_16x16x4(kf[kt][s], bq[s], sacc[kt]);
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float sv = (kt < nkt && kt * 16 + 4 * g + i < kk) ? sacc[kt][i] * a.scale : -INFINITY;
        sacc[kt][i] = sv;
        mx = fmaxf(mx, sv);
      }
    }
    mx = cross_rows_max(mx);
    float z = 0.0f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = __expf(sacc[kt][i] - mx);
        sacc[kt][i] = e;
        z += e;
      }
    z = cross_rows_sum(z);
    const float f = mh / z;
    v4f oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = v4f{0.f, 0.f, 0.f, 0.f};
    if constexpr (sizeof(T) == 2) {
      // exact bf16 values, P in two bf16 parts (mfma_weights); slots of tiles kt and
      // kt + 1 form one product over 32 (k = 8 g + j: slot 4 g + j of tile kt
      // for j < 4, of tile kt + 1 otherwise); a missing tile contributes 0
#pragma unroll
      for (int kt = 0; kt < NKT; kt += 2) {
        if (kt >= nkt) break;
        float p8[8];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int i = 0; i < 4; ++i) p8[4 * h + i] = (kt + h < NKT && kt + h < nkt) ? sacc[min(kt + h, NKT - 1)][i] * f : 0.0f;
        const Split8 ps = split8(p8);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          float v8[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            v8[i] = vf[kt][i][dt];
            v8[4 + i] = kt + 1 < NKT ? vf[min(kt + 1, NKT - 1)][i][dt] : 0.0f;
          }
          oacc[dt] = mfma_weights<bf16_t>(v8, ps, oacc[dt]);
        }
      }
    } else {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        if (kt < nkt) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float pv = sacc[kt][i] * f;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) oacc[dt] = mfma_f32_16x16x4(vf[kt][i][dt], pv, oacc[dt]);
          }
        }
      }
    }
    float o[4 * DT];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[i * DT + dt] = oacc[dt][i] + vbs[wave][DT * 4 * g + i * DT + dt];
    buf_store<4 * DT>(ro, row0 >= 0 ? static_cast<uint32_t>(row0) * D * ESZ + DT * 4 * g * ESZ : kNone, 0, o, T{});
    row0 = row1;
    row1 = row2;
    if constexpr (PF) {
#pragma unroll
      for (int s = 0; s < KS; ++s) bq[s] = bqn[s];
    }
  }
}

// ---------------------------------------------------------------------------
// Host launchers.
// ---------------------------------------------------------------------------
template <int D, typename T>
static hipError_t launch_centroids_t(const Problem& p, const Workspace& ws, hipStream_t s) {
  constexpr int per_block = 4 * (64 / D);  // clusters per workgroup
  hipLaunchKernelGGL((centroid_kernel<D, T>), dim3((p.C + per_block - 1) / per_block, p.units()),
                     dim3(256), 0, s,
                     static_cast<const T*>(p.q), ws.sizes, ws.offsets, ws.members, p.n, p.C, ws.qc);
  return hipGetLastError();
}

// Compute units of the current device (cached per device; 0 if unknown).
static int device_cus() {
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
  return cus[dev] > 0 ? cus[dev] : 0;
}

template <int D, typename T>
static hipError_t launch_coop_centroids_t(const Problem& p, const Workspace& ws, hipStream_t s) {
  constexpr int per_block = 4 * (64 / D);  // items per workgroup of the final sums (and of VL = 1)
  constexpr int per_block4 = 4 * (256 / D);  // items per workgroup of the block sums with VL = 4
  const int nwg = (p.n + ws.coop_q - 1) / ws.coop_q;
  if (!ws.coop_sums) {
    const long long n1 = static_cast<long long>(p.units()) * nwg * p.C;
    // four dimensions per lane once that still leaves eight waves per compute
    // unit (sweep point 23.7 -> 22.1 us in fp32, 23.9 -> 19.5 us in bf16; at
    // N = 8192 its 800 waves took 15.1 us against 12.6 us with one)
    const int cus = device_cus();
    if (cus > 0 && n1 / (per_block4 / 4) >= 8LL * cus)
      hipLaunchKernelGGL((centroid_part_kernel<D, T, 4>), dim3(static_cast<unsigned>((n1 + per_block4 - 1) / per_block4)),
                         dim3(256), 0, s, static_cast<const T*>(p.q), ws.members, ws.cbases, ws.clsizes,
                         p.n, p.C, nwg, n1, ws.qc_part);
    else
      hipLaunchKernelGGL((centroid_part_kernel<D, T, 1>), dim3(static_cast<unsigned>((n1 + per_block - 1) / per_block)),
                         dim3(256), 0, s, static_cast<const T*>(p.q), ws.members, ws.cbases, ws.clsizes,
                         p.n, p.C, nwg, n1, ws.qc_part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const long long n2 = static_cast<long long>(p.units()) * p.C;
  hipLaunchKernelGGL((centroid_final_kernel<D>), dim3(static_cast<unsigned>((n2 + per_block - 1) / per_block)),
                     dim3(256), 0, s, ws.qc_part, ws.sizes, p.C, nwg, n2, ws.qc);
  return hipGetLastError();
}

hipError_t launch_coop_centroids(const Problem& p, const Workspace& ws, hipStream_t s) {
  if (p.d == 32)
    return p.dtype == 0 ? launch_coop_centroids_t<32, float>(p, ws, s) : launch_coop_centroids_t<32, bf16_t>(p, ws, s);
  return p.dtype == 0 ? launch_coop_centroids_t<64, float>(p, ws, s) : launch_coop_centroids_t<64, bf16_t>(p, ws, s);
}

hipError_t launch_centroids(const Problem& p, const Workspace& ws, hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_centroids_t<32, float>(p, ws, s) : launch_centroids_t<32, bf16_t>(p, ws, s);
  return p.dtype == 0 ? launch_centroids_t<64, float>(p, ws, s) : launch_centroids_t<64, bf16_t>(p, ws, s);
}

static AttnArgs make_args(const Problem& p, const Workspace& ws, const int32_t* topk_in) {
  AttnArgs a;
  a.assign = ws.assign;
  a.qc = ws.qc;
  a.sizes = ws.sizes;
  a.offsets = ws.offsets;
  a.members = ws.members;
  a.q = p.q;
  a.k = p.k;
  a.v = p.v;
  a.lengths = p.lengths;
  a.heads = p.heads;
  a.N = p.n;
  a.C = p.C;
  a.nchunk = ws.nchunk;
  a.ntile = (p.C + 15) / 16;
  a.ncg = (p.C + 3) / 4;
  a.pchunk = kChunk;
  a.npc = 1;
  // at most C + n / kSparseChunk (cluster, member chunk) items per unit
  a.nsg = (p.C + (p.n + kSparseChunk - 1) / kSparseChunk + 3) / 4;
  a.units = p.units();
  a.topk = p.topk > 0 ? p.topk : 1;
  a.scale = 1.0f / sqrtf(static_cast<float>(p.d));
  a.topk_in = topk_in;
  a.pm = ws.pm;
  a.pz = ws.pz;
  a.pacc = ws.pacc;
  a.cand_idx = ws.cand_idx;
  a.cand_val = ws.cand_val;
  a.topk_out = ws.topk;
  a.mass = ws.mass;
  a.vcb = ws.vcb;
  a.stats = ws.stats;
  a.out = p.out;
  return a;
}

// Key tiles of the register-resident sparse routine (k <= 16 * NKT).
static int sparse_tiles(int topk) { return topk <= 16 ? 1 : topk <= 32 ? 2 : topk <= 64 ? 4 : 8; }

// part 0: the tile kernel (single chunk: the whole stage); part 1: the merge
// of several chunks (nothing for a single chunk).  The clustered variant
// takes every chunk in the single-pass kernel, flash_chunk keys per
// workgroup.
// Keys per workgroup of the clustered partial pass over several chunks:
// 2 kFlashChunk when that grid still covers 80 % of two workgroups per
// compute unit (fewer, longer workgroups: the length-sweep point's clustered
// stage 100.7 -> 96.7 us in fp32, 60.1 -> 57.0 us in bf16), else
// kFlashChunk (a grid of a quarter of the chip at 2 kFlashChunk ran 50 %
// slower).  A multiple of kChunk, so the partial states keep their stride.
static int flash_chunk(const Problem& p, int ntile) {
  const int cus = device_cus();
  constexpr int big = 2 * kFlashChunk;
  const long long wgs = static_cast<long long>((p.n + big - 1) / big) * ntile * p.units();
  return cus > 0 && 5 * wgs >= 8LL * cus ? big : kFlashChunk;
}

template <int D, typename T>
static hipError_t launch_attn_t(const Problem& p, const Workspace& ws, const int32_t* topk_in,
                                int part, hipStream_t s) {
  AttnArgs a = make_args(p, ws, topk_in);
  const bool improved = p.topk > 0;
  const dim3 g2(xcd_grid(static_cast<long long>(a.ncg) * a.units));
  if (ws.nchunk == 1) {
    if (part != 0) return hipSuccess;
    const dim3 g1(xcd_grid(static_cast<long long>(a.ntile) * a.units));
    if (improved)
      hipLaunchKernelGGL((attn_tile_kernel<D, T, 1>), g1, dim3(kTileThreads), 0, s, a);
    else
      hipLaunchKernelGGL((attn_flash_kernel<D, T, false>), g1, dim3(kFlashThreads), 0, s, a);
    return hipGetLastError();
  }
  if (!improved) {
    a.pchunk = flash_chunk(p, a.ntile);  // the states keep the stride ws.nchunk
    a.npc = (p.n + a.pchunk - 1) / a.pchunk;
    if (part == 0) {
      const dim3 g1(xcd_grid(static_cast<long long>(a.npc) * a.ntile * a.units));
      hipLaunchKernelGGL((attn_flash_kernel<D, T, true>), g1, dim3(kFlashThreads), 0, s, a);
    } else {
      hipLaunchKernelGGL((attn_merge_kernel<D, T, false>), g2, dim3(256), 0, s, a);
    }
    return hipGetLastError();
  }
  const dim3 g1(xcd_grid(static_cast<long long>(a.nchunk) * a.ntile * a.units));
  if (part == 0)
    hipLaunchKernelGGL((attn_tile_kernel<D, T, 3>), g1, dim3(kTileThreads), 0, s, a);
  else
    hipLaunchKernelGGL((attn_merge_kernel<D, T, true>), g2, dim3(256), 0, s, a);
  return hipGetLastError();
}

// The per-query improved values run as their own kernel: their gathers of the
// T rows want many waves in flight, which the LDS-heavy tile kernel cannot
// offer.
template <int D, typename T>
static hipError_t launch_sparse_t(const Problem& p, const Workspace& ws, hipStream_t s) {
  const AttnArgs a = make_args(p, ws, nullptr);
  const dim3 g2(xcd_grid(static_cast<long long>(a.nsg) * a.units));
  switch (sparse_tiles(p.topk)) {
    case 1: hipLaunchKernelGGL((sparse_kernel<D, T, 1>), g2, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((sparse_kernel<D, T, 2>), g2, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((sparse_kernel<D, T, 4>), g2, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((sparse_kernel<D, T, 8>), g2, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

// Oracle-top: the improved top-k search on the query rows themselves (C = n
// rows per unit), each output row from its own T.
template <int D, typename T>
static hipError_t launch_otop_t(const Problem& p, const Workspace& ws, hipStream_t s) {
  const AttnArgs a = make_args(p, ws, nullptr);
  const dim3 g1(xcd_grid(static_cast<long long>(a.nchunk) * a.ntile * a.units));
  if (ws.nchunk == 1) {
    hipLaunchKernelGGL((attn_tile_kernel<D, T, 4>), g1, dim3(kTileThreads), 0, s, a);
    return hipGetLastError();
  }
  const dim3 g2(xcd_grid(static_cast<long long>(a.ncg) * a.units));
  hipLaunchKernelGGL((attn_tile_kernel<D, T, 5>), g1, dim3(kTileThreads), 0, s, a);
  hipLaunchKernelGGL((attn_merge_kernel<D, T, true, true>), g2, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_oracle_top(const Problem& p, const Workspace& ws, hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_otop_t<32, float>(p, ws, s) : launch_otop_t<32, bf16_t>(p, ws, s);
  return p.dtype == 0 ? launch_otop_t<64, float>(p, ws, s) : launch_otop_t<64, bf16_t>(p, ws, s);
}

// Centroid attention: softmax statistics, values (and, clustered in one key
// chunk, the output rows via Eq. (6)); improved: top-k, mass and rest part.
hipError_t launch_centroid_attention(const Problem& p, const Workspace& ws, const int32_t* topk_in,
                                     int part, hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_attn_t<32, float>(p, ws, topk_in, part, s) : launch_attn_t<32, bf16_t>(p, ws, topk_in, part, s);
  return p.dtype == 0 ? launch_attn_t<64, float>(p, ws, topk_in, part, s) : launch_attn_t<64, bf16_t>(p, ws, topk_in, part, s);
}

// Improved values of every member query (Section 3.3).
hipError_t launch_sparse(const Problem& p, const Workspace& ws, hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_sparse_t<32, float>(p, ws, s) : launch_sparse_t<32, bf16_t>(p, ws, s);
  return p.dtype == 0 ? launch_sparse_t<64, float>(p, ws, s) : launch_sparse_t<64, bf16_t>(p, ws, s);
}

}  // namespace ca
