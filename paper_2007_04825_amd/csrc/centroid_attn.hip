// Centroids (Eq. 3), centroid attention (Eqs. 4-5) and the top-k keys of
// each cluster with their attention mass (Section 3.3).
//
// centroid_kernel: one wave per cluster sums the member rows of Q in fp64
//   (members in ascending query order) and divides by the cluster size.
//
// centroid_attn_partial_kernel: one workgroup per (unit, 16 centroids,
//   1024-key chunk).  Logits S^T = K Q^c^T come from v_mfma_f32_16x16x4f32
//   with keys as rows and centroids as columns; they are scaled by 1/sqrt(d),
//   masked past the valid length and kept in LDS, so A^c is never written to
//   HBM.  Per centroid the chunk's row maximum m, sum z = sum exp(s - m), and
//   (improved variant) the chunk's top-k candidates are taken from LDS; then
//   V^T P^T accumulates the unnormalised chunk values on the matrix cores.
//   The result layout of the first product is exactly the B-operand layout of
//   the second (key 4*g + i of a 16-key tile sits in lane group g, register
//   i), so P never leaves registers between the two products.
//
// centroid_attn_merge_kernel: one wave per cluster merges the chunks with the
//   log-sum-exp rule, giving V^c = A^c V; for the improved variant it selects
//   T_j among the chunk candidates, computes m_j = sum_{T_j} A^c and the rest
//   part V^b_j = V^c_j - sum_{T_j} A^c_jl V_l.
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
  constexpr int RPS = 64 / D;  // member rows per step
  const int u = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = blockIdx.x * 4 + wave;
  if (j >= C) return;
  const int sz = sizes[static_cast<size_t>(u) * C + j];
  float* dst = qc + (static_cast<size_t>(u) * C + j) * D;
  const int t = lane % D, r = lane / D;
  if (sz == 0) {
    if (lane < D) dst[lane] = 0.0f;
    return;
  }
  const int32_t* mem = members + static_cast<size_t>(u) * N + offsets[static_cast<size_t>(u) * (C + 1) + j];
  const T* qu = q + static_cast<size_t>(u) * N * D;
  double acc = 0.0;
#pragma unroll 4
  for (int m = r; m < sz; m += RPS) acc += static_cast<double>(to_f32(qu[static_cast<size_t>(mem[m]) * D + t]));
  if (RPS == 2) acc += __shfl_xor(acc, 32);
  if (lane < D) dst[t] = static_cast<float>(acc / static_cast<double>(sz));
}

// ---------------------------------------------------------------------------
// Eqs. (4)-(5) per chunk of keys.
// ---------------------------------------------------------------------------
constexpr int kLStride = kChunk + 4;  // floats per LDS logit row

template <int D, typename T, bool TOPK>
__global__ __launch_bounds__(256) void centroid_attn_partial_kernel(
    const float* __restrict__ qc, const int32_t* __restrict__ sizes, const T* __restrict__ kmat,
    const T* __restrict__ vmat, const int32_t* __restrict__ lengths, int heads, int N, int C,
    int nchunk, int topk, float scale, float* __restrict__ pm, float* __restrict__ pz,
    float* __restrict__ pacc, int32_t* __restrict__ cand_idx, float* __restrict__ cand_val) {
  __shared__ float logits[16 * kLStride];
  __shared__ float rowm[16], rowz[16];
  __shared__ int hist[4][256];
  __shared__ int selpos[4][128];
  __shared__ int any_nonempty;
  const int chunk = blockIdx.x, tile = blockIdx.y, u = blockIdx.z;
  const int n = unit_length(lengths, u / heads, N);
  const int k0 = chunk * kChunk;
  if (k0 >= n) return;
  const int kn = min(kChunk, n - k0);
  const int j0 = tile * 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) any_nonempty = 0;
  __syncthreads();
  if (tid < 16 && j0 + tid < C && sizes[static_cast<size_t>(u) * C + j0 + tid] > 0) any_nonempty = 1;
  __syncthreads();
  if (!any_nonempty) return;

  const int c = lane & 15, g = lane >> 4;
  constexpr int KS = D / 4;  // reduction steps of the 16x16x4 product
  // B operand: centroid c, dimensions g*KS .. g*KS+KS-1.
  float bq[KS];
  if (j0 + c < C) {
    load_row<KS>(qc + (static_cast<size_t>(u) * C + j0 + c) * D + g * KS, bq);
  } else {
#pragma unroll
    for (int s = 0; s < KS; ++s) bq[s] = 0.0f;
  }
  const T* ku = kmat + (static_cast<size_t>(u) * N + k0) * D;
  const T* vu = vmat + (static_cast<size_t>(u) * N + k0) * D;
  const int nkt = (kn + 15) / 16;

  // logits of this chunk
  for (int kt = wave; kt < nkt; kt += 4) {
    const int key = kt * 16 + c;  // A operand row
    float a[KS];
    if (key < kn) {
      load_row<KS>(ku + static_cast<size_t>(key) * D + g * KS, a);
    } else {
#pragma unroll
      for (int s = 0; s < KS; ++s) a[s] = 0.0f;
    }
    v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) acc = mfma_f32_16x16x4(a[s], bq[s], acc);
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = (kt * 16 + 4 * g + i < kn) ? acc[i] * scale : -INFINITY;
    *reinterpret_cast<float4*>(&logits[c * kLStride + kt * 16 + 4 * g]) = make_float4(o[0], o[1], o[2], o[3]);
  }
  __syncthreads();

  // per-row maximum, sum and top-k candidates (wave w owns rows 4w..4w+3)
  const int kk = min(topk, kn);
  for (int rr = 0; rr < 4; ++rr) {
    const int r = wave * 4 + rr;
    const float* row = &logits[r * kLStride];
    float mx = -INFINITY;
    for (int x = lane; x < kn; x += 64) mx = fmaxf(mx, row[x]);
    mx = wave_max(mx);
    float z = 0.0f;
    for (int x = lane; x < kn; x += 64) z += __expf(row[x] - mx);
    z = wave_sum(z);
    if (lane == 0) {
      rowm[r] = mx;
      rowz[r] = z;
    }
    if (TOPK && j0 + r < C) {
      const int got = wave_select_topk([&](int pos) { return order_key(row[pos]); }, kn, kk,
                                       hist[wave], selpos[wave]);
      wave_lds_sync();
      const size_t cb = ((static_cast<size_t>(u) * C + j0 + r) * nchunk + chunk) * topk;
      for (int x = lane; x < topk; x += 64) {
        const bool ok = x < got;
        const int pos = ok ? selpos[wave][x] : 0;
        cand_idx[cb + x] = ok ? k0 + pos : -1;
        cand_val[cb + x] = ok ? row[pos] : -INFINITY;
      }
      wave_lds_sync();
    }
  }
  __syncthreads();

  // unnormalised chunk values: O^T = V^T P^T, P = exp(S - m)
  constexpr int DT = D / 16;
  v4f oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = v4f{0.f, 0.f, 0.f, 0.f};
  const float mc = rowm[c];
  for (int kt = wave; kt < nkt; kt += 4) {
    const float4 s4 = *reinterpret_cast<const float4*>(&logits[c * kLStride + kt * 16 + 4 * g]);
    const float p[4] = {__expf(s4.x - mc), __expf(s4.y - mc), __expf(s4.z - mc), __expf(s4.w - mc)};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = kt * 16 + 4 * g + i;
      const bool ok = key < kn;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const float a = ok ? to_f32(vu[static_cast<size_t>(key) * D + 16 * dt + c]) : 0.0f;
        oacc[dt] = mfma_f32_16x16x4(a, p[i], oacc[dt]);
      }
    }
  }
  __syncthreads();  // logits no longer needed: reuse them for the cross-wave sum
  float* red = logits;  // [4 waves][16 centroids][D]
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
    *reinterpret_cast<float4*>(&red[(wave * 16 + c) * D + 16 * dt + 4 * g]) =
        make_float4(oacc[dt][0], oacc[dt][1], oacc[dt][2], oacc[dt][3]);
  __syncthreads();
  for (int x = tid; x < 16 * D; x += 256) {
    const int cc = x / D, dim = x % D;
    if (j0 + cc >= C) continue;
    const float sum = ((red[(0 * 16 + cc) * D + dim] + red[(1 * 16 + cc) * D + dim]) +
                       red[(2 * 16 + cc) * D + dim]) + red[(3 * 16 + cc) * D + dim];
    const size_t pj = (static_cast<size_t>(u) * C + j0 + cc) * nchunk + chunk;
    pacc[pj * D + dim] = sum;
    if (dim == 0) {
      pm[pj] = rowm[cc];
      pz[pj] = rowz[cc];
    }
  }
}

// ---------------------------------------------------------------------------
// Merge of the chunks, top-k set, mass and rest part.
// ---------------------------------------------------------------------------
template <int D, typename T, bool TOPK>
__global__ __launch_bounds__(256) void centroid_attn_merge_kernel(
    const float* __restrict__ qc, const int32_t* __restrict__ sizes, const T* __restrict__ kmat,
    const T* __restrict__ vmat, const int32_t* __restrict__ lengths, int heads, int N, int C,
    int nchunk, int topk, float scale, const float* __restrict__ pm, const float* __restrict__ pz,
    const float* __restrict__ pacc, const int32_t* __restrict__ cand_idx,
    const float* __restrict__ cand_val, const int32_t* __restrict__ topk_in,
    int32_t* __restrict__ topk_out, float* __restrict__ mass, float* __restrict__ vcb) {
  __shared__ int hist[4][256];
  __shared__ int selpos[4][128];
  __shared__ float selval[4][128];
  __shared__ float vcs[4][D];
  const int u = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = blockIdx.x * 4 + wave;
  if (j >= C) return;
  const size_t uj = static_cast<size_t>(u) * C + j;
  const int sz = sizes[uj];
  if (sz == 0) {
    for (int x = lane; x < D; x += 64) vcb[uj * D + x] = 0.0f;
    if (TOPK) {
      for (int x = lane; x < topk; x += 64) topk_out[uj * topk + x] = -1;
      if (lane == 0) mass[uj] = 0.0f;
    }
    return;
  }
  const int n = unit_length(lengths, u / heads, N);
  const int nch = (n + kChunk - 1) / kChunk;
  const float* pmj = pm + uj * nchunk;
  const float* pzj = pz + uj * nchunk;
  float M = -INFINITY;
  for (int x = lane; x < nch; x += 64) M = fmaxf(M, pmj[x]);
  M = wave_max(M);
  float Z = 0.0f;
  for (int x = lane; x < nch; x += 64) Z += pzj[x] * __expf(pmj[x] - M);
  Z = wave_sum(Z);
  // V^c = sum_chunks exp(m_c - M) acc_c / Z   (lane -> dimension)
  constexpr int RPS = 64 / D;
  const int t = lane % D, r = lane / D;
  float acc = 0.0f;
  for (int x = r; x < nch; x += RPS) acc += __expf(pmj[x] - M) * pacc[(uj * nchunk + x) * D + t];
  if (RPS == 2) acc += __shfl_xor(acc, 32);
  const float vc = acc / Z;
  if (!TOPK) {
    if (lane < D) vcb[uj * D + t] = vc;
    return;
  }
  if (lane < D) vcs[wave][t] = vc;
  const int kk = min(topk, n);
  int cnt;
  if (topk_in != nullptr) {
    // caller-supplied set: entries until the first negative one; logits recomputed
    const int32_t* tin = topk_in + uj * topk;
    const float* qj = qc + uj * D;
    const T* ku = kmat + static_cast<size_t>(u) * N * D;
    cnt = 0;
    while (cnt < topk && tin[cnt] >= 0 && tin[cnt] < n) ++cnt;
    for (int x = lane; x < cnt; x += 64) {
      const int key = tin[x];
      float dot = 0.0f;
      for (int d = 0; d < D; ++d) dot = fmaf(qj[d], to_f32(ku[static_cast<size_t>(key) * D + d]), dot);
      selpos[wave][x] = key;
      selval[wave][x] = dot * scale;
    }
  } else if (nch == 1) {
    cnt = kk;
    const size_t cb = uj * nchunk * topk;
    for (int x = lane; x < kk; x += 64) {
      selpos[wave][x] = cand_idx[cb + x];
      selval[wave][x] = cand_val[cb + x];
    }
  } else {
    const int32_t* ci = cand_idx + uj * nchunk * topk;
    const float* cv = cand_val + uj * nchunk * topk;
    const int m = nch * topk;
    cnt = wave_select_topk([&](int pos) { return ci[pos] >= 0 ? order_key(cv[pos]) : 0u; }, m, kk,
                           hist[wave], selpos[wave]);
    wave_lds_sync();
    for (int x = lane; x < cnt; x += 64) {
      const int pos = selpos[wave][x];
      selval[wave][x] = cv[pos];
    }
    wave_lds_sync();
    for (int x = lane; x < cnt; x += 64) selpos[wave][x] = ci[selpos[wave][x]];
  }
  wave_lds_sync();
  // m_j and the top-k part of A^c V
  float msum = 0.0f;
  for (int x = lane; x < cnt; x += 64) msum += __expf(selval[wave][x] - M) / Z;
  msum = wave_sum(msum);
  const T* vu = vmat + static_cast<size_t>(u) * N * D;
  float top = 0.0f;
  for (int x = r; x < cnt; x += RPS) {
    const float w = __expf(selval[wave][x] - M) / Z;
    top += w * to_f32(vu[static_cast<size_t>(selpos[wave][x]) * D + t]);
  }
  if (RPS == 2) top += __shfl_xor(top, 32);
  if (lane < D) vcb[uj * D + t] = vcs[wave][t] - top;
  for (int x = lane; x < topk; x += 64) topk_out[uj * topk + x] = x < cnt ? selpos[wave][x] : -1;
  if (lane == 0) mass[uj] = msum;
}

// ---------------------------------------------------------------------------
// Host launchers.
// ---------------------------------------------------------------------------
template <int D, typename T>
static hipError_t launch_centroids_t(const Problem& p, const Workspace& ws, hipStream_t s) {
  hipLaunchKernelGGL((centroid_kernel<D, T>), dim3((p.C + 3) / 4, p.units()), dim3(256), 0, s,
                     static_cast<const T*>(p.q), ws.sizes, ws.offsets, ws.members, p.n, p.C, ws.qc);
  return hipGetLastError();
}

hipError_t launch_centroids(const Problem& p, const Workspace& ws, hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_centroids_t<32, float>(p, ws, s) : launch_centroids_t<32, bf16_t>(p, ws, s);
  return p.dtype == 0 ? launch_centroids_t<64, float>(p, ws, s) : launch_centroids_t<64, bf16_t>(p, ws, s);
}

template <int D, typename T, bool TOPK>
static hipError_t launch_cattn_t(const Problem& p, const Workspace& ws, const int32_t* topk_in,
                                 hipStream_t s) {
  const float scale = 1.0f / sqrtf(static_cast<float>(D));
  const int tk = TOPK ? p.topk : 1;
  dim3 g1(ws.nchunk, (p.C + 15) / 16, p.units());
  hipLaunchKernelGGL((centroid_attn_partial_kernel<D, T, TOPK>), g1, dim3(256), 0, s, ws.qc,
                     ws.sizes, static_cast<const T*>(p.k), static_cast<const T*>(p.v), p.lengths,
                     p.heads, p.n, p.C, ws.nchunk, tk, scale, ws.pm, ws.pz, ws.pacc, ws.cand_idx,
                     ws.cand_val);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g2((p.C + 3) / 4, p.units());
  hipLaunchKernelGGL((centroid_attn_merge_kernel<D, T, TOPK>), g2, dim3(256), 0, s, ws.qc, ws.sizes,
                     static_cast<const T*>(p.k), static_cast<const T*>(p.v), p.lengths, p.heads,
                     p.n, p.C, ws.nchunk, tk, scale, ws.pm, ws.pz, ws.pacc, ws.cand_idx,
                     ws.cand_val, topk_in, ws.topk, ws.mass, ws.vcb);
  return hipGetLastError();
}

template <int D, typename T>
static hipError_t launch_cattn_d(const Problem& p, const Workspace& ws, const int32_t* topk_in,
                                 hipStream_t s) {
  return p.topk > 0 ? launch_cattn_t<D, T, true>(p, ws, topk_in, s)
                    : launch_cattn_t<D, T, false>(p, ws, topk_in, s);
}

hipError_t launch_centroid_attention(const Problem& p, const Workspace& ws, const int32_t* topk_in,
                                     hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_cattn_d<32, float>(p, ws, topk_in, s) : launch_cattn_d<32, bf16_t>(p, ws, topk_in, s);
  return p.dtype == 0 ? launch_cattn_d<64, float>(p, ws, topk_in, s) : launch_cattn_d<64, bf16_t>(p, ws, topk_in, s);
}

}  // namespace ca
