// Backward pass of clustered and improved-clustered attention.
//
// The paper trains through the operator but writes no backward pass; the
// partition (the K-means assignment of Section 3.2.2) and the top-k sets of
// Section 3.3 are discrete and are held constant.  The gradient then flows
// through the centroids (Eq. 3), the centroid softmax (Eqs. 4-5), the
// broadcast (Eq. 6) and, for the improved variant, through the exact top-k
// logits, the mass m_j and the rest part V^b_j of the supplementary
// decomposition.  With g_i the output gradient of query i and G_j the sum of
// g_i over the members of cluster j:
//
//   clustered:   gA_jl = G_j . V_l,  dV_l += sum_j A^c_jl G_j
//   improved:    gA_jl = dm_j (l in T_j), G_j . V_l (otherwise),
//                dV_l += sum_j [l not in T_j] A^c_jl G_j, plus the top-k part
//                (w_i = softmax_T(q_i k_l / sqrt d), U_i = w_i V_T):
//                dm_j = sum_i g_i . U_i,  gt_il = m_j w_il (g_i . V_l - g_i . U_i),
//                dQ_i += gt_i K_T / sqrt d,  dK_l += sum_i gt_il Q_i / sqrt d,
//                dV_l += m_j sum_i w_il g_i
//   both:        dS_jl = A^c_jl (gA_jl - delta_j),  delta_j = sum_l A^c_jl gA_jl
//                (clustered: G_j . V^c_j; improved: m_j dm_j + G_j . V^b_j),
//                dQ^c_j = sum_l dS_jl K_l / sqrt d,  dK_l += sum_j dS_jl Q^c_j / sqrt d,
//                dQ_i += dQ^c_{a_i} / |S_{a_i}|.
//
// Kernels (all on the caller's stream, in this order):
//   bwd_cluster_sums_kernel (clustered) / bwd_sparse_kernel (improved): G_j,
//     delta_j (and dm_j); the improved one also writes the top-k part of dQ
//     and per-cluster partial key and value gradients of its T_j rows.
//   bwd_tile_kernel: one workgroup per (unit, block of 128 keys) loops over
//     the 16-centroid tiles: A^c from the logits and the forward's softmax
//     statistics, gA and dS on the fp32 matrix cores; dK and dV of the block
//     accumulate in registers, dQ^c leaves one partial per key block.
//   bwd_dqc_reduce_kernel, bwd_dq_kernel: dQ^c over the key blocks in order,
//     then dQ_i.
//   improved only: bwd_index_kernel (first) gives every entry (j, r) of the
//     top-k sets a slot in a per-unit list ordered by key; bwd_sparse_kernel
//     writes the partial key/value gradient row of the entry into that slot,
//     so each key's partials lie together, and bwd_index_gather_kernel adds
//     them into dK and dV as 64-bit fixed-point integers, whose sum does not
//     depend on the order of the slots.  No floating-point atomics: the
//     result is deterministic.
#include <limits.h>
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "select.h"

namespace ca {

constexpr int kBwdKeys = 128;  // keys per workgroup of bwd_tile_kernel
constexpr int kBwdWaves = 8;   // waves per workgroup of bwd_tile_kernel (one key tile each)
constexpr int kIdxKeys = 8192;  // keys per workgroup of bwd_index_kernel

struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* dout;
  const int32_t* lengths;
  int heads, N, C, topk, nkb, units;
  float scale;
  // state left by the forward pass
  const int32_t* assign;
  const int32_t* sizes;
  const int32_t* offsets;
  const int32_t* members;
  const float* qc;
  const float* stats;
  const int32_t* tsets;
  const float* mass;
  const float* vcb;
  // backward scratch and results
  float* G;         // [U][C][D]
  float* delta;     // [U][C]
  float* dm;        // [U][C]
  float* dqc_part;  // [U][nkb][C][D]
  float* dqc;       // [U][C][D]
  float* part_k;    // [U][C * topk][D] rows in key order: slot epos[j * topk + r]
  float* part_v;    // [U][C * topk][D]
  int32_t* icnt;    // [U][N]  entries per key
  int32_t* ioff;    // [U][N]  first slot of each key (the unit's entries in key order)
  int32_t* epos;    // [U][C * topk] slot of entry (j, r) with T_j[r] = key
  float* dq;
  float* dk;
  float* dv;
};

// Sum over the D lanes of a lane group (D = 32: two groups per wave).
template <int D>
__device__ __forceinline__ float dgroup_sum(float x) {
  x = row16_sum(x);
  x += lane_xor16(x);
  if constexpr (D == 64) x += lane_xor32(x);
  return x;
}

// ---------------------------------------------------------------------------
// Clustered: G_j = sum of the members' output gradients (member order) and
// delta_j = G_j . V^c_j.  D lanes per cluster (lane = dimension).
// ---------------------------------------------------------------------------
template <int D, typename T>
__global__ __launch_bounds__(256) void bwd_cluster_sums_kernel(BwdArgs a) {
  constexpr int GPW = 64 / D;
  const int u = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = (blockIdx.x * 4 + wave) * GPW + lane / D;
  const int t = lane % D;
  const int C = a.C;
  const bool ok = j < C;
  const size_t uj = static_cast<size_t>(u) * C + (ok ? j : 0);
  const int sz = ok ? a.sizes[uj] : 0;
  const int32_t* mem = a.members + static_cast<size_t>(u) * a.N + (ok ? a.offsets[static_cast<size_t>(u) * (C + 1) + j] : 0);
  const T* gu = static_cast<const T*>(a.dout) + static_cast<size_t>(u) * a.N * D;
  const float vb = a.vcb[uj * D + t];
  // members in batches of eight, every load issued (positions past the
  // cluster read its last member again and are not added), added in order
  float acc = 0.0f;
  for (int m = 0; m < sz; m += 8) {
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = to_f32(gu[static_cast<size_t>(mem[min(m + e, sz - 1)]) * D + t]);
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (m + e < sz) acc += x[e];
  }
  const float del = dgroup_sum<D>(sz > 0 ? acc * vb : 0.0f);
  if (ok) {
    a.G[uj * D + t] = acc;
    if (t == 0) a.delta[uj] = del;
  }
}

// ---------------------------------------------------------------------------
// Improved: top-k part of the gradient, one wave per cluster.  The cluster's
// T rows of K and V are staged in LDS; member queries go 16 at a time:
//   t^T  = K_T Q^T,  gv^T = V_T g^T        (keys as rows, queries as columns)
//   w = softmax over the slots, rho_i = sum_l w_il gv_il = g_i . U_i
//   gt = m_j w (gv - rho)
//   dQ_i  (top-k part) = gt_i K_T / sqrt d  (written to dq)
//   dK_T += gt^T Q / sqrt d,  dV_T += m_j w^T g  (LDS accumulators; the
//   products over the queries take w and gt transposed through LDS)
// and G_j = sum g_i, dm_j = sum_i rho_i, delta_j = m_j dm_j + G_j . V^b_j.
// ---------------------------------------------------------------------------
template <int D, int NKT>
struct SparseBwdShared {
  static constexpr int KP = 16 * NKT;
  static constexpr int DP = D + 4;
  float k[KP][DP];
  float v[KP][DP];
  float acck[KP][D];
  float accv[KP][D];
  float q[16][DP];
  float g[16][DP];
  float wt[KP][17];
  float gtt[KP][17];
  int tp[KP];
  int ep[KP];  // slots of the partial rows
};

template <int D, typename T, int NKT>
__global__ __launch_bounds__(64) void bwd_sparse_kernel(BwdArgs a) {
  constexpr int KS = D / 4, DT = D / 16, KP = 16 * NKT;
  constexpr uint32_t ESZ = sizeof(T);
  constexpr uint32_t kNone = 0x80000000u;
  __shared__ SparseBwdShared<D, NKT> sh;
  const int wi = xcd_work_item();  // cluster fastest, then (batch, head)
  if (wi >= a.C * a.units) return;
  const int u = wi / a.C, j = wi % a.C;
  const int lane = threadIdx.x, c = lane & 15, g = lane >> 4;
  const int C = a.C;
  const size_t uj = static_cast<size_t>(u) * C + j;
  // everything that depends on the cluster alone is requested at once: its
  // size, offset and mass, its T entries with their partial-row slots (the
  // slots of entries past T are read and ignored) and V^b_j
  const int sz = a.sizes[uj];
  const int off = a.offsets[static_cast<size_t>(u) * (C + 1) + j];
  const float mh = a.mass[uj];
  constexpr int TR = (KP + 63) / 64;
  int keyv[TR], epv[TR];
#pragma unroll
  for (int r = 0; r < TR; ++r) {
    const int x = 64 * r + lane;
    const size_t at = uj * a.topk + min(x, a.topk - 1);
    keyv[r] = x < a.topk ? a.tsets[at] : -1;
    epv[r] = a.epos[at];
  }
  float vcbl[KS];
#pragma unroll
  for (int s2 = 0; s2 < KS; ++s2) vcbl[s2] = a.vcb[uj * D + g * KS + s2];
  if (sz == 0) {
    for (int x = lane; x < D; x += 64) a.G[uj * D + x] = 0.0f;
    if (lane == 0) {
      a.delta[uj] = 0.0f;
      a.dm[uj] = 0.0f;
    }
    return;
  }
  // T: the leading non-negative entries
  int kk = 0;
#pragma unroll
  for (int r = 0; r < TR; ++r) {
    const int x = 64 * r + lane;
    if (x < KP) {
      sh.tp[x] = keyv[r];
      sh.ep[x] = keyv[r] >= 0 ? epv[r] : 0;
    }
    kk += __popcll(__ballot(keyv[r] >= 0));
  }
  const int nkt = (kk + 15) >> 4;
  const size_t base = static_cast<size_t>(u) * a.N * D;
  const uint32_t ubytes = static_cast<uint32_t>(a.N) * D * ESZ;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(static_cast<const T*>(a.q) + base, ubytes);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(static_cast<const T*>(a.k) + base, ubytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(static_cast<const T*>(a.v) + base, ubytes);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(static_cast<const T*>(a.dout) + base, ubytes);
  wave_lds_sync();
  // T rows of K and V into LDS (rows past kk are zero); 4 lanes per row, up
  // to four 16-row groups requested before any is stored
  constexpr int RL = D / 4;  // values per lane
  constexpr int RG = KP / 16 < 4 ? KP / 16 : 4;  // row groups in flight
  for (int r0 = 0; r0 < KP; r0 += 16 * RG) {
    float kx[RG][RL], vx[RG][RL];
#pragma unroll
    for (int q = 0; q < RG; ++q) {
      const int r = r0 + 16 * q + (lane >> 2), part = lane & 3;
      const uint32_t vo = r < kk ? static_cast<uint32_t>(sh.tp[r]) * D * ESZ + part * RL * ESZ : kNone;
      buf_load<RL>(rk, vo, 0, kx[q], T{});
      buf_load<RL>(rv, vo, 0, vx[q], T{});
    }
#pragma unroll
    for (int q = 0; q < RG; ++q) {
      const int r = r0 + 16 * q + (lane >> 2), part = lane & 3;
#pragma unroll
      for (int e = 0; e < RL; ++e) {
        sh.k[r][part * RL + e] = kx[q][e];
        sh.v[r][part * RL + e] = vx[q][e];
      }
    }
  }
  for (int x = lane; x < KP * D; x += 64) {
    sh.acck[x / D][x % D] = 0.0f;
    sh.accv[x / D][x % D] = 0.0f;
  }
  const int32_t* mem = a.members + static_cast<size_t>(u) * a.N + off;
  // member index of row lane / 4 of the next member tile, requested one tile
  // ahead (positions past the cluster read its last member and are ignored)
  int qnext = mem[min(lane >> 2, sz - 1)];
  float gsum[KS];  // per lane: sum over its query column of g, dims g * KS ..
#pragma unroll
  for (int s = 0; s < KS; ++s) gsum[s] = 0.0f;
  float dmacc = 0.0f;
  const uint32_t orow = static_cast<uint32_t>(D) * ESZ;
  for (int mt = 0; mt < sz; mt += 16) {
    // member rows of Q and of the output gradient into LDS
    int qrow;  // member index of row lane / 4 of this tile, -1 past the cluster
    {
      const int r = lane >> 2, part = lane & 3;
      const int qi = mt + r < sz ? qnext : -1;
      qrow = qi;
      const uint32_t vo = qi >= 0 ? static_cast<uint32_t>(qi) * orow + part * RL * ESZ : kNone;
      float qx[RL], gx[RL];
      buf_load<RL>(rq, vo, 0, qx, T{});
      buf_load<RL>(rg, vo, 0, gx, T{});
      qnext = mem[min(mt + 16 + r, sz - 1)];
#pragma unroll
      for (int e = 0; e < RL; ++e) {
        sh.q[r][part * RL + e] = qx[e];
        sh.g[r][part * RL + e] = gx[e];
      }
    }
    wave_lds_sync();
    const bool qvalid = mt + c < sz;
    float bq[KS], bg[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      bq[s] = sh.q[c][g * KS + s];
      bg[s] = sh.g[c][g * KS + s];
      gsum[s] += bg[s];
    }
    v4f t[NKT], gv[NKT];
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
      t[kt] = v4f{0.f, 0.f, 0.f, 0.f};
      gv[kt] = v4f{0.f, 0.f, 0.f, 0.f};
      if (kt < nkt) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          t[kt] = mfma_f32_16x16x4(sh.k[kt * 16 + c][g * KS + s], bq[s], t[kt]);
          gv[kt] = mfma_f32_16x16x4(sh.v[kt * 16 + c][g * KS + s], bg[s], gv[kt]);
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float sv = (kt < nkt && kt * 16 + 4 * g + i < kk) ? t[kt][i] * a.scale : -INFINITY;
        t[kt][i] = sv;
        mx = fmaxf(mx, sv);
      }
    }
    mx = cross_rows_max(mx);
    float z = 0.0f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = __expf(t[kt][i] - mx);
        t[kt][i] = e;
        z += e;
      }
    z = cross_rows_sum(z);
    const float rz = 1.0f / z;
    float rho = 0.0f;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        t[kt][i] *= rz;  // w
        rho += t[kt][i] * gv[kt][i];
      }
    rho = cross_rows_sum(rho);
    if (g == 0 && qvalid) dmacc += rho;
    // gt = m w (gv - rho); w is scaled by m for dV_T; both zero for invalid queries
    v4f gt[NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        gt[kt][i] = qvalid ? mh * t[kt][i] * (gv[kt][i] - rho) : 0.0f;
        t[kt][i] = qvalid ? mh * t[kt][i] : 0.0f;
      }
    // top-k part of dQ: O^T = K_T^T gt^T (lane: query c, dims DT*4g ..)
    {
      v4f oq[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oq[dt] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        if (kt < nkt) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
              oq[dt] = mfma_f32_16x16x4(sh.k[kt * 16 + 4 * g + i][DT * c + dt], gt[kt][i], oq[dt]);
        }
      }
      float o[4 * DT];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[i * DT + dt] = oq[dt][i] * a.scale;
      const int qs = __shfl(qrow, 4 * c);  // row c's index, from lane 4 c (every lane active)
      const int qi = qvalid ? qs : -1;
      if (qi >= 0) {
        float* dst = a.dq + base + static_cast<size_t>(qi) * D + DT * 4 * g;
#pragma unroll
        for (int x = 0; x < 4 * DT; x += 4) *reinterpret_cast<float4*>(dst + x) = make_float4(o[x], o[x + 1], o[x + 2], o[x + 3]);
      }
    }
    // w and gt transposed to [slot][query]
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sh.wt[kt * 16 + 4 * g + i][c] = t[kt][i];
        sh.gtt[kt * 16 + 4 * g + i][c] = gt[kt][i];
      }
    wave_lds_sync();
    // dK_T += gt^T Q, dV_T += (m w)^T g: rows = slots, columns = dims, k = queries
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
      if (kt >= nkt) continue;
      v4f rk[DT], rv[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) rk[dt] = rv[dt] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const float ak = sh.gtt[kt * 16 + c][4 * s + g];
        const float av = sh.wt[kt * 16 + c][4 * s + g];
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          rk[dt] = mfma_f32_16x16x4(ak, sh.q[4 * s + g][16 * dt + c], rk[dt]);
          rv[dt] = mfma_f32_16x16x4(av, sh.g[4 * s + g][16 * dt + c], rv[dt]);
        }
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sh.acck[kt * 16 + 4 * g + i][16 * dt + c] += rk[dt][i];
          sh.accv[kt * 16 + 4 * g + i][16 * dt + c] += rv[dt][i];
        }
    }
    wave_lds_sync();
  }
  // G_j (lanes of group g hold dims g * KS ..), dm_j, delta_j
  float gvb = 0.0f;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    gsum[s] = row16_sum(gsum[s]);
    gvb += gsum[s] * vcbl[s];
  }
  gvb = cross_rows_sum(gvb);
  const float dmj = wave_sum(dmacc);
  if (c == 0) {
#pragma unroll
    for (int s = 0; s < KS; ++s) a.G[uj * D + g * KS + s] = gsum[s];
  }
  if (lane == 0) {
    a.dm[uj] = dmj;
    a.delta[uj] = mh * dmj + gvb;
  }
  // partial key and value gradients of the T rows, each into its key's slot
  float* pk = a.part_k + static_cast<size_t>(u) * C * a.topk * D;
  float* pv = a.part_v + static_cast<size_t>(u) * C * a.topk * D;
  constexpr int LPR = D / 4;  // lanes per row, four dims each
  for (int x = lane; x < kk * LPR; x += 64) {
    const int r = x / LPR, c4 = (x % LPR) * 4;
    const size_t at = static_cast<size_t>(sh.ep[r]) * D + c4;
    const float4 k4 = *reinterpret_cast<const float4*>(&sh.acck[r][c4]);
    *reinterpret_cast<float4*>(pk + at) = make_float4(k4.x * a.scale, k4.y * a.scale, k4.z * a.scale, k4.w * a.scale);
    *reinterpret_cast<float4*>(pv + at) = *reinterpret_cast<const float4*>(&sh.accv[r][c4]);
  }
}

// ---------------------------------------------------------------------------
// Centroid part, one workgroup per (unit, block of kBwdKeys keys); wave w owns
// key tile w of the block and loops over the 16-centroid tiles.
//   S^T = K Q^c^T and gA^T = V G^T (keys as rows, centroids as columns), P^T
//   from the forward's row maximum and normaliser, dS^T = P^T (gA^T - delta);
//   dQ^c^T += K^T dS^T (one partial per key block, summed over the waves);
//   dV += P^T G and dK += dS^T Q^c over the centroids, with P and dS
//   transposed through LDS.  Improved: gA = dm_j on the keys of T_j, and P is
//   masked there for dV (those keys' value gradient is the top-k part's).
// ---------------------------------------------------------------------------
template <int D>
struct TileBwdShared {
  static constexpr int DP = D + 4;
  float qc[2][16][DP];
  float g[2][16][DP];
  float st[2][16][4];              // row maximum, 1 / normaliser, delta, dm
  int valid[2][16];
  float red[kBwdWaves][16][D];     // per-wave dQ^c partials of the current tile
  float pt[kBwdWaves][16][17];     // P^T of the wave's key tile, [key][centroid]
  float dst[kBwdWaves][16][17];    // dS^T
  uint32_t tmask[256][kBwdKeys / 32];  // improved: key l of the block is in T_j
};

template <int D, typename T, bool IMPROVED>
__global__ __launch_bounds__(64 * kBwdWaves) void bwd_tile_kernel(BwdArgs a) {
  constexpr int KS = D / 4, DT = D / 16;
  constexpr uint32_t ESZ = sizeof(T);
  __shared__ TileBwdShared<D> sh;
  const int wi = xcd_work_item();  // key block fastest, then (batch, head)
  if (wi >= a.nkb * a.units) return;
  const int kb = wi % a.nkb, u = wi / a.nkb;
  const int n = unit_length(a.lengths, u / a.heads, a.N);
  const int k0 = kb * kBwdKeys;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int C = a.C;
  const size_t base = static_cast<size_t>(u) * a.N * D;
  const int kn = min(kBwdKeys, n - k0);  // valid keys of the block (may be <= 0)
  if (kn <= 0) {
    // a block past the length: zero gradients for its rows
    for (int x = tid; x < kBwdKeys * D; x += 64 * kBwdWaves) {
      const int row = k0 + x / D;
      if (row < a.N) {
        a.dk[base + static_cast<size_t>(row) * D + x % D] = 0.0f;
        a.dv[base + static_cast<size_t>(row) * D + x % D] = 0.0f;
      }
    }
    return;
  }
  const T* ku = static_cast<const T*>(a.k) + base + static_cast<size_t>(k0) * D;
  const T* vu = static_cast<const T*>(a.v) + base + static_cast<size_t>(k0) * D;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(ku, static_cast<uint32_t>(kn) * D * ESZ);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vu, static_cast<uint32_t>(kn) * D * ESZ);
  // key tile rows of this wave in the three operand layouts
  float kA[KS], vA[KS], kT[4][DT];
  buf_load<KS>(rk, ((wave * 16 + c) * D + g * KS) * ESZ, 0, kA, T{});
  buf_load<KS>(rv, ((wave * 16 + c) * D + g * KS) * ESZ, 0, vA, T{});
#pragma unroll
  for (int i = 0; i < 4; ++i) buf_load<DT>(rk, ((wave * 16 + 4 * g + i) * D + DT * c) * ESZ, 0, kT[i], T{});

  const int ntile = (C + 15) / 16;
  // a centroid tile's rows of Q^c and G, and its statistics, go through
  // registers: requested (stage_load) before the previous tile goes through
  // the products, written to LDS buffer jt & 1 (stage_store) after it, so
  // that their latency overlaps the products
  constexpr int NTH = 64 * kBwdWaves;
  constexpr int EPT = (16 * D + NTH - 1) / NTH;  // row elements per thread
  struct Stage {
    float qc[EPT], g[EPT];
    int sz[EPT];
    float st[4];
    int szs;
  };
  auto stage_load = [&](int jt, Stage& r) {
    const int j0 = jt * 16;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int x = tid + e * NTH;
      const int cc = min(x / D, 15), dim = x % D, j = min(j0 + cc, C - 1);
      const size_t uj = static_cast<size_t>(u) * C + j;
      r.sz[e] = a.sizes[uj];
      r.qc[e] = a.qc[uj * D + dim];
      r.g[e] = a.G[uj * D + dim];
    }
    if (tid < 16) {
      const size_t uj = static_cast<size_t>(u) * C + min(j0 + tid, C - 1);
      r.szs = a.sizes[uj];
      r.st[0] = a.stats[uj * 2];
      r.st[1] = a.stats[uj * 2 + 1];
      r.st[2] = a.delta[uj];
      r.st[3] = IMPROVED ? a.dm[uj] : 0.0f;
    }
  };
  auto stage_store = [&](int jt, const Stage& r) {
    const int b = jt & 1, j0 = jt * 16;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int x = tid + e * NTH;
      if (EPT * NTH == 16 * D || x < 16 * D) {
        const int cc = x / D, dim = x % D;
        const bool ok = j0 + cc < C && r.sz[e] > 0;
        sh.qc[b][cc][dim] = ok ? r.qc[e] : 0.0f;
        sh.g[b][cc][dim] = ok ? r.g[e] : 0.0f;
      }
    }
    if (tid < 16) {
      const bool ok = j0 + tid < C && r.szs > 0;
      sh.valid[b][tid] = ok;
      sh.st[b][tid][0] = ok ? r.st[0] : 0.0f;
      sh.st[b][tid][1] = ok ? 1.0f / r.st[1] : 0.0f;
      sh.st[b][tid][2] = ok ? r.st[2] : 0.0f;
      sh.st[b][tid][3] = (ok && IMPROVED) ? r.st[3] : 0.0f;
    }
  };
  Stage pre;
  stage_load(0, pre);
  if constexpr (IMPROVED) {
    for (int x = tid; x < ntile * 16 * (kBwdKeys / 32); x += NTH) sh.tmask[x / (kBwdKeys / 32)][x % (kBwdKeys / 32)] = 0u;
    __syncthreads();
    // (the top-k lists of empty clusters are not defined); eight entries per
    // thread requested together with their cluster sizes
    const int tot = C * a.topk;
    const int32_t* ts = a.tsets + static_cast<size_t>(u) * C * a.topk;
    const int32_t* szu = a.sizes + static_cast<size_t>(u) * C;
    for (int x0 = 0; x0 < tot; x0 += 8 * NTH) {
      int key[8], sz[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int x = min(x0 + tid + e * NTH, tot - 1);
        key[e] = ts[x];
        sz[e] = szu[x / a.topk];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int x = x0 + tid + e * NTH;
        const int j = x / a.topk;
        if (x < tot && sz[e] > 0 && key[e] >= k0 && key[e] < k0 + kBwdKeys)
          atomicOr(&sh.tmask[j][(key[e] - k0) >> 5], 1u << ((key[e] - k0) & 31));
      }
    }
  }
  stage_store(0, pre);
  __syncthreads();

  v4f dkacc[DT], dvacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) dkacc[dt] = dvacc[dt] = v4f{0.f, 0.f, 0.f, 0.f};
  for (int jt = 0; jt < ntile; ++jt) {
    const int b = jt & 1, j0 = jt * 16;
    if (jt + 1 < ntile) stage_load(jt + 1, pre);  // in flight during the products
    {
      float bq[KS], bg[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        bq[s] = sh.qc[b][c][g * KS + s];
        bg[s] = sh.g[b][c][g * KS + s];
      }
      v4f sacc = {0.f, 0.f, 0.f, 0.f}, gacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        sacc = mfma_f32_16x16x4(kA[s], bq[s], sacc);
        gacc = mfma_f32_16x16x4(vA[s], bg[s], gacc);
      }
      const float mc = sh.st[b][c][0], rzc = sh.st[b][c][1], delc = sh.st[b][c][2], dmc = sh.st[b][c][3];
      const bool cval = sh.valid[b][c] != 0;
      float ds[4], pv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int l = wave * 16 + 4 * g + i;  // key within the block
        const bool ok = cval && l < kn;
        const float p = ok ? __expf(sacc[i] * a.scale - mc) * rzc : 0.0f;
        float ga = gacc[i];
        bool in_t = false;
        if constexpr (IMPROVED) in_t = ok && ((sh.tmask[j0 + c][l >> 5] >> (l & 31)) & 1u);
        if (in_t) ga = dmc;
        ds[i] = p * (ga - delc);
        pv[i] = in_t ? 0.0f : p;
      }
      // this wave's part of dQ^c^T for the tile
      v4f dq4[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) dq4[dt] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) dq4[dt] = mfma_f32_16x16x4(kT[i][dt], ds[i], dq4[dt]);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 4; ++r) sh.red[wave][c][DT * (4 * g + r) + dt] = dq4[dt][r];
      // P and dS transposed: rows = keys, columns = centroids
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sh.pt[wave][4 * g + i][c] = pv[i];
        sh.dst[wave][4 * g + i][c] = ds[i];
      }
      wave_lds_sync();
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const float ap = sh.pt[wave][c][4 * s + g];
        const float ad = sh.dst[wave][c][4 * s + g];
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          dvacc[dt] = mfma_f32_16x16x4(ap, sh.g[b][4 * s + g][16 * dt + c], dvacc[dt]);
          dkacc[dt] = mfma_f32_16x16x4(ad, sh.qc[b][4 * s + g][16 * dt + c], dkacc[dt]);
        }
      }
    }
    __syncthreads();
    // dQ^c partial of the tile (summed over the waves in order), next tile staged
    for (int x = tid; x < 16 * D; x += 64 * kBwdWaves) {
      const int cc = x / D, dim = x % D;
      float sacc = 0.0f;
#pragma unroll
      for (int w = 0; w < kBwdWaves; ++w) sacc += sh.red[w][cc][dim];
      if (j0 + cc < C) a.dqc_part[((static_cast<size_t>(u) * a.nkb + kb) * C + j0 + cc) * D + dim] = sacc * a.scale;
    }
    if (jt + 1 < ntile) stage_store(jt + 1, pre);
    __syncthreads();
  }
  // dK and dV of the wave's keys (rows past the length get 0)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = k0 + wave * 16 + 4 * g + i;
    if (row >= a.N) continue;
    const bool ok = row < n;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      a.dk[base + static_cast<size_t>(row) * D + 16 * dt + c] = ok ? dkacc[dt][i] * a.scale : 0.0f;
      a.dv[base + static_cast<size_t>(row) * D + 16 * dt + c] = ok ? dvacc[dt][i] : 0.0f;
    }
  }
}

// dQ^c_j = (sum over the key blocks, in order, of the partials) / |S_j|.
template <int D>
__global__ __launch_bounds__(256) void bwd_dqc_reduce_kernel(BwdArgs a) {
  constexpr int Q4 = D / 4;  // four consecutive dimensions per thread
  const size_t x = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  const size_t total = static_cast<size_t>(a.units) * a.C * Q4;
  if (x >= total) return;
  const int d4 = static_cast<int>(x % Q4);
  const size_t uj = x / Q4;
  const int u = static_cast<int>(uj / a.C), j = static_cast<int>(uj % a.C);
  const int sz = a.sizes[uj];
  const int n = unit_length(a.lengths, u / a.heads, a.N);
  const int nkbv = (n + kBwdKeys - 1) / kBwdKeys;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (sz > 0)
    for (int kb = 0; kb < nkbv; ++kb) {
      const float4 t =
          reinterpret_cast<const float4*>(a.dqc_part)[((static_cast<size_t>(u) * a.nkb + kb) * a.C + j) * Q4 + d4];
      s.x += t.x;
      s.y += t.y;
      s.z += t.z;
      s.w += t.w;
    }
  const float fsz = static_cast<float>(sz);
  reinterpret_cast<float4*>(a.dqc)[uj * Q4 + d4] =
      sz > 0 ? make_float4(s.x / fsz, s.y / fsz, s.z / fsz, s.w / fsz) : make_float4(0.f, 0.f, 0.f, 0.f);
}

// dQ_i = dQ^c_{a_i} (+ the top-k part already in dq for the improved variant);
// rows past the length get 0.  Four consecutive dimensions per thread.
template <int D, bool IMPROVED>
__global__ __launch_bounds__(256) void bwd_dq_kernel(BwdArgs a) {
  constexpr int Q4 = D / 4;
  const size_t x = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;  // float4 index
  const size_t total = static_cast<size_t>(a.units) * a.N * Q4;
  if (x >= total) return;
  const int d4 = static_cast<int>(x % Q4);
  const size_t ui = x / Q4;
  const int u = static_cast<int>(ui / a.N), i = static_cast<int>(ui % a.N);
  const int n = unit_length(a.lengths, u / a.heads, a.N);
  float4* dq4 = reinterpret_cast<float4*>(a.dq) + x;
  if (i >= n) {
    *dq4 = make_float4(0.f, 0.f, 0.f, 0.f);
    return;
  }
  const int j = min(max(a.assign[ui], 0), a.C - 1);
  const float4 cp = reinterpret_cast<const float4*>(a.dqc)[(static_cast<size_t>(u) * a.C + j) * Q4 + d4];
  if constexpr (IMPROVED) {
    const float4 t = *dq4;
    *dq4 = make_float4(t.x + cp.x, t.y + cp.y, t.z + cp.z, t.w + cp.w);
  } else {
    *dq4 = cp;
  }
}

// ---------------------------------------------------------------------------
// Inverse index of the top-k sets (improved): one workgroup per unit walks
// its keys in ranges of kIdxKeys.  Per range: counts per key (LDS atomics,
// order-free), an exclusive prefix sum continuing the previous ranges' total,
// then every entry takes a slot of its key.  The slots of one key are
// consecutive; their order among the key's entries is not fixed (the
// gather's sum does not depend on it).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void bwd_index_kernel(BwdArgs a) {
  __shared__ int cnt[kIdxKeys];
  __shared__ int off[kIdxKeys];
  __shared__ int wsum[16];
  const int u = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = unit_length(a.lengths, u / a.heads, a.N);
  const int C = a.C, K = a.topk;
  const int32_t* ts = a.tsets + static_cast<size_t>(u) * C * K;
  const int32_t* sz = a.sizes + static_cast<size_t>(u) * C;
  int32_t* icu = a.icnt + static_cast<size_t>(u) * a.N;
  int32_t* iou = a.ioff + static_cast<size_t>(u) * a.N;
  int32_t* ep = a.epos + static_cast<size_t>(u) * C * K;
  int base = 0;  // slots taken by the earlier ranges
  for (int lo = 0; lo < n; lo += kIdxKeys) {
    const int hi = min(n, lo + kIdxKeys);
    for (int x = tid; x < kIdxKeys; x += 1024) cnt[x] = 0;
    __syncthreads();
    for (int x = tid; x < C * K; x += 1024) {
      if (sz[x / K] == 0) continue;  // no list for an empty cluster
      const int key = ts[x];
      if (key >= lo && key < hi) atomicAdd(&cnt[key - lo], 1);
    }
    __syncthreads();
    // exclusive prefix sum of cnt[0 .. hi - lo), 8 keys per thread
    const int m = hi - lo;
    int local[kIdxKeys / 1024], tot = 0;
#pragma unroll
    for (int e = 0; e < kIdxKeys / 1024; ++e) {
      const int x = tid * (kIdxKeys / 1024) + e;
      local[e] = x < m ? cnt[x] : 0;
      tot += local[e];
    }
    const int incl = wave_incl_scan(tot);
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int run = base + incl - tot, total = 0;
    for (int w = 0; w < 16; ++w) {
      if (w < wave) run += wsum[w];
      total += wsum[w];
    }
#pragma unroll
    for (int e = 0; e < kIdxKeys / 1024; ++e) {
      const int x = tid * (kIdxKeys / 1024) + e;
      if (x < m) {
        off[x] = run;
        icu[lo + x] = local[e];
        iou[lo + x] = run;
        cnt[x] = 0;  // now the fill cursor
      }
      run += local[e];
    }
    __syncthreads();
    for (int x = tid; x < C * K; x += 1024) {
      if (sz[x / K] == 0) continue;
      const int key = ts[x];
      if (key >= lo && key < hi) ep[x] = off[key - lo] + atomicAdd(&cnt[key - lo], 1);
    }
    base += total;
    __syncthreads();  // before the next range clears the tables
  }
}

// dK_l and dV_l receive the top-k parts of the entries of key l: one thread
// per (key, four dimensions) adds the partial rows as 64-bit fixed-point
// integers (2^-32 units; integer addition is exact and associative, so the
// order of the entries does not matter and the result is deterministic),
// then rounds the sum once into fp32.  A term is converted exactly when
// |x| >= 2^-8 (x * 2^32 is then an integer in fp32) and to the nearest unit
// otherwise.  Terms up to |x| = 2^22 are held, so no sum of at most 256 of
// them leaves the int64 range; a larger or non-finite term is not added but
// sets `bad`, and the entry it belongs to is written as NaN, so that the
// caller sees it instead of a silently altered sum.
__device__ __forceinline__ long long to_fixed32(float x, bool& bad) {
  const bool ok = fabsf(x) <= 4194304.0f;  // false for NaN as well
  bad = bad || !ok;
  return ok ? __float2ll_rn(x * 4294967296.0f) : 0ll;
}
template <int D>
__global__ __launch_bounds__(256) void bwd_index_gather_kernel(BwdArgs a) {
  constexpr int Q4 = D / 4;
  const size_t x = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  if (x >= static_cast<size_t>(a.units) * a.N * Q4) return;
  const int part = static_cast<int>(x % Q4);
  const size_t ul = x / Q4;
  const int u = static_cast<int>(ul / a.N), key = static_cast<int>(ul % a.N);
  const int n = unit_length(a.lengths, u / a.heads, a.N);
  if (key >= n) return;
  const int cnt = a.icnt[ul];
  if (cnt == 0) return;
  // the key's partial rows are the consecutive slots ioff .. ioff + cnt - 1
  const size_t first = static_cast<size_t>(u) * a.C * a.topk + a.ioff[ul];
  const float4* pk = reinterpret_cast<const float4*>(a.part_k) + first * Q4 + part;
  const float4* pv = reinterpret_cast<const float4*>(a.part_v) + first * Q4 + part;
  long long ak[4] = {0, 0, 0, 0}, av[4] = {0, 0, 0, 0};
  bool bk[4] = {false, false, false, false}, bv[4] = {false, false, false, false};
  constexpr int B = 4;  // entries in flight (consecutive rows)
  for (int t0 = 0; t0 < cnt; t0 += B) {
    float4 k4[B], v4[B];
#pragma unroll
    for (int t = 0; t < B; ++t) {
      const bool ok = t0 + t < cnt;
      k4[t] = ok ? pk[static_cast<size_t>(t0 + t) * Q4] : make_float4(0.f, 0.f, 0.f, 0.f);
      v4[t] = ok ? pv[static_cast<size_t>(t0 + t) * Q4] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int t = 0; t < B; ++t) {
      ak[0] += to_fixed32(k4[t].x, bk[0]); ak[1] += to_fixed32(k4[t].y, bk[1]);
      ak[2] += to_fixed32(k4[t].z, bk[2]); ak[3] += to_fixed32(k4[t].w, bk[3]);
      av[0] += to_fixed32(v4[t].x, bv[0]); av[1] += to_fixed32(v4[t].y, bv[1]);
      av[2] += to_fixed32(v4[t].z, bv[2]); av[3] += to_fixed32(v4[t].w, bv[3]);
    }
  }
  constexpr double kUnit = 1.0 / 4294967296.0;
  float4* dk4 = reinterpret_cast<float4*>(a.dk) + ul * Q4 + part;
  float4* dv4 = reinterpret_cast<float4*>(a.dv) + ul * Q4 + part;
  float4 sk = *dk4, sv = *dv4;
  auto add = [&](float base, long long sum, bool bad) {
    return bad ? __builtin_nanf("") : static_cast<float>(static_cast<double>(base) + static_cast<double>(sum) * kUnit);
  };
  sk.x = add(sk.x, ak[0], bk[0]);
  sk.y = add(sk.y, ak[1], bk[1]);
  sk.z = add(sk.z, ak[2], bk[2]);
  sk.w = add(sk.w, ak[3], bk[3]);
  sv.x = add(sv.x, av[0], bv[0]);
  sv.y = add(sv.y, av[1], bv[1]);
  sv.z = add(sv.z, av[2], bv[2]);
  sv.w = add(sv.w, av[3], bv[3]);
  *dk4 = sk;
  *dv4 = sv;
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
int bwd_key_blocks(int n) { return (n + kBwdKeys - 1) / kBwdKeys; }

static int sparse_bwd_tiles(int topk) { return topk <= 16 ? 1 : topk <= 32 ? 2 : topk <= 64 ? 4 : 8; }

template <int D, typename T>
static hipError_t launch_backward_t(const BwdProblem& p, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  BwdArgs a;
  a.q = p.q;
  a.k = p.k;
  a.v = p.v;
  a.dout = p.dout;
  a.lengths = p.lengths;
  a.heads = p.heads;
  a.N = p.n;
  a.C = p.C;
  a.topk = p.topk > 0 ? p.topk : 1;
  a.nkb = bwd_key_blocks(p.n);
  a.units = p.batch * p.heads;
  a.scale = 1.0f / sqrtf(static_cast<float>(D));
  a.assign = p.fws->assign;
  a.sizes = p.fws->sizes;
  a.offsets = p.fws->offsets;
  a.members = p.fws->members;
  a.qc = p.fws->qc;
  a.stats = p.fws->stats;
  a.tsets = p.fws->topk;
  a.mass = p.fws->mass;
  a.vcb = p.fws->vcb;
  a.G = p.bws.G;
  a.delta = p.bws.delta;
  a.dm = p.bws.dm;
  a.dqc_part = p.bws.dqc_part;
  a.dqc = p.bws.dqc;
  a.part_k = p.bws.part_k;
  a.part_v = p.bws.part_v;
  a.icnt = p.bws.icnt;
  a.ioff = p.bws.ioff;
  a.epos = p.bws.epos;
  a.dq = p.dq;
  a.dk = p.dk;
  a.dv = p.dv;
  const bool improved = p.topk > 0;
  const long long U = a.units;
  auto blocks = [](long long count) { return dim3(static_cast<unsigned>((count + 255) / 256)); };
  hipError_t e;
  if (improved) {
    hipLaunchKernelGGL(bwd_index_kernel, dim3(static_cast<unsigned>(U)), dim3(1024), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 gs(xcd_grid(static_cast<long long>(p.C) * U));
    switch (sparse_bwd_tiles(p.topk)) {
      case 1: hipLaunchKernelGGL((bwd_sparse_kernel<D, T, 1>), gs, dim3(64), 0, s, a); break;
      case 2: hipLaunchKernelGGL((bwd_sparse_kernel<D, T, 2>), gs, dim3(64), 0, s, a); break;
      case 4: hipLaunchKernelGGL((bwd_sparse_kernel<D, T, 4>), gs, dim3(64), 0, s, a); break;
      default: hipLaunchKernelGGL((bwd_sparse_kernel<D, T, 8>), gs, dim3(64), 0, s, a); break;
    }
  } else {
    constexpr int per_block = 4 * (64 / D);
    hipLaunchKernelGGL((bwd_cluster_sums_kernel<D, T>), dim3((p.C + per_block - 1) / per_block, static_cast<unsigned>(U)),
                       dim3(256), 0, s, a);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const dim3 gt(xcd_grid(static_cast<long long>(a.nkb) * U));
  if (ev0 && (e = hipEventRecord(ev0, s)) != hipSuccess) return e;
  if (improved)
    hipLaunchKernelGGL((bwd_tile_kernel<D, T, true>), gt, dim3(64 * kBwdWaves), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_tile_kernel<D, T, false>), gt, dim3(64 * kBwdWaves), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (ev1 && (e = hipEventRecord(ev1, s)) != hipSuccess) return e;
  hipLaunchKernelGGL((bwd_dqc_reduce_kernel<D>), blocks(U * p.C * (D / 4)), dim3(256), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (improved)
    hipLaunchKernelGGL((bwd_dq_kernel<D, true>), blocks(U * p.n * (D / 4)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_dq_kernel<D, false>), blocks(U * p.n * (D / 4)), dim3(256), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (improved) {
    hipLaunchKernelGGL((bwd_index_gather_kernel<D>), blocks(U * p.n * (D / 4)), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_backward(const BwdProblem& p, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (p.d == 32)
    return p.dtype == 0 ? launch_backward_t<32, float>(p, s, ev0, ev1) : launch_backward_t<32, bf16_t>(p, s, ev0, ev1);
  return p.dtype == 0 ? launch_backward_t<64, float>(p, s, ev0, ev1) : launch_backward_t<64, bf16_t>(p, s, ev0, ev1);
}

}  // namespace ca
