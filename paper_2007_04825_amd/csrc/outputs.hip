// Output stages.
//
// broadcast_kernel (clustered, Eq. 6): every valid query row receives V^c of
//   its cluster; padded rows receive 0.  One float4 of a row per thread, so
//   the writes are fully coalesced.
//
// sparse_kernel (improved, Section 3.3 and the supplementary decomposition):
//   one wave per cluster.  K and V rows of T_j are gathered into LDS once;
//   the members are then processed 16 at a time: S^T = K_T Q^T on the matrix
//   cores (keys as rows, queries as columns), a softmax over the k_eff keys of
//   each query column scaled by m_j, and O^T = V_T^T P^T, again with P taken
//   straight from the result registers of the first product.  The rest part
//   V^b_j is added and the rows are scattered back to their query positions.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "select.h"

namespace ca {

template <int D, typename T>
__global__ __launch_bounds__(256) void broadcast_kernel(const int32_t* __restrict__ assign,
                                                        const float* __restrict__ vc,
                                                        const int32_t* __restrict__ lengths,
                                                        int heads, int N, int C,
                                                        T* __restrict__ out) {
  constexpr int PR = D / 4;  // float4 parts per row
  const int u = blockIdx.y;
  const int n = unit_length(lengths, u / heads, N);
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int row = idx / PR, part = idx % PR;
  if (row >= N) return;
  T* o = out + (static_cast<size_t>(u) * N + row) * D + part * 4;
  if (row < n) {
    const int a = assign[static_cast<size_t>(u) * N + row];
    const float4 x = *reinterpret_cast<const float4*>(vc + (static_cast<size_t>(u) * C + a) * D + part * 4);
    store4(o, x.x, x.y, x.z, x.w);
  } else {
    store4(o, 0.f, 0.f, 0.f, 0.f);
  }
}

template <int D, typename T>
__global__ __launch_bounds__(256) void pad_zero_kernel(const int32_t* __restrict__ lengths,
                                                       int heads, int N, T* __restrict__ out) {
  constexpr int PR = D / 4;
  const int u = blockIdx.y;
  const int n = unit_length(lengths, u / heads, N);
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int row = idx / PR, part = idx % PR;
  if (row >= N || row < n) return;
  store4(out + (static_cast<size_t>(u) * N + row) * D + part * 4, 0.f, 0.f, 0.f, 0.f);
}

constexpr int kMaxKTiles = 8;  // k <= 128

template <int D, typename T>
__global__ __launch_bounds__(256) void sparse_kernel(
    const T* __restrict__ q, const T* __restrict__ kmat, const T* __restrict__ vmat,
    const int32_t* __restrict__ lengths, int heads, int N, int C, int topk, int kpad,
    float scale, const int32_t* __restrict__ sizes, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ members, const int32_t* __restrict__ topk_g,
    const float* __restrict__ mass, const float* __restrict__ vb, T* __restrict__ out) {
  extern __shared__ float smem[];
  constexpr int KST = D + 4;  // LDS row stride of K_T
  constexpr int KS = D / 4;
  constexpr int DT = D / 16;
  const int wpb = blockDim.x >> 6;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int u = blockIdx.y, j = blockIdx.x * wpb + wave;
  if (j >= C) return;
  const size_t uj = static_cast<size_t>(u) * C + j;
  const int sz = sizes[uj];
  if (sz == 0) return;
  const int n = unit_length(lengths, u / heads, N);
  const int kk = min(topk, n);
  const int nkt = (kk + 15) / 16;
  float* KT = smem + static_cast<size_t>(wave) * kpad * (KST + D);
  float* VT = KT + kpad * KST;
  const int32_t* tj = topk_g + uj * topk;
  const T* ku = kmat + static_cast<size_t>(u) * N * D;
  const T* vu = vmat + static_cast<size_t>(u) * N * D;
  for (int x = lane; x < kpad * D; x += 64) {
    const int r = x / D, t = x % D;
    const int key = r < kk ? tj[r] : -1;
    const bool ok = key >= 0 && key < n;
    KT[r * KST + t] = ok ? to_f32(ku[static_cast<size_t>(key) * D + t]) : 0.0f;
    VT[r * D + t] = ok ? to_f32(vu[static_cast<size_t>(key) * D + t]) : 0.0f;
  }
  const float mh = mass[uj];
  const int c = lane & 15, g = lane >> 4;
  float4 vbv[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) vbv[dt] = *reinterpret_cast<const float4*>(vb + uj * D + 16 * dt + 4 * g);
  const int32_t* mem = members + static_cast<size_t>(u) * N + offsets[static_cast<size_t>(u) * (C + 1) + j];
  const T* qu = q + static_cast<size_t>(u) * N * D;
  T* ou = out + static_cast<size_t>(u) * N * D;
  wave_lds_sync();

  for (int mt = 0; mt < sz; mt += 16) {
    const int mi = mt + c;
    const int row = mi < sz ? mem[mi] : -1;
    float bq[KS];
    if (row >= 0) {
      load_row<KS>(qu + static_cast<size_t>(row) * D + g * KS, bq);
    } else {
#pragma unroll
      for (int s = 0; s < KS; ++s) bq[s] = 0.0f;
    }
    v4f sacc[kMaxKTiles];
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < kMaxKTiles; ++kt) {
      sacc[kt] = v4f{0.f, 0.f, 0.f, 0.f};
      if (kt < nkt) {
        const float* ar = KT + (kt * 16 + c) * KST + g * KS;
#pragma unroll
        for (int s = 0; s < KS; ++s) sacc[kt] = mfma_f32_16x16x4(ar[s], bq[s], sacc[kt]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float sv = (kt * 16 + 4 * g + i < kk) ? sacc[kt][i] * scale : -INFINITY;
          sacc[kt][i] = sv;
          mx = fmaxf(mx, sv);
        }
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    float z = 0.0f;
#pragma unroll
    for (int kt = 0; kt < kMaxKTiles; ++kt) {
      if (kt < nkt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = __expf(sacc[kt][i] - mx);
          sacc[kt][i] = e;
          z += e;
        }
      }
    }
    z += __shfl_xor(z, 16);
    z += __shfl_xor(z, 32);
    const float f = mh / z;
    v4f oacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < kMaxKTiles; ++kt) {
      if (kt < nkt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pv = sacc[kt][i] * f;
          const float* vr = VT + (kt * 16 + 4 * g + i) * D + c;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) oacc[dt] = mfma_f32_16x16x4(vr[16 * dt], pv, oacc[dt]);
        }
      }
    }
    if (row >= 0) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        store4(ou + static_cast<size_t>(row) * D + 16 * dt + 4 * g, oacc[dt][0] + vbv[dt].x,
               oacc[dt][1] + vbv[dt].y, oacc[dt][2] + vbv[dt].z, oacc[dt][3] + vbv[dt].w);
    }
  }
}

// ---------------------------------------------------------------------------
// Host launchers.
// ---------------------------------------------------------------------------
template <int D, typename T>
static hipError_t launch_broadcast_t(const Problem& p, const int32_t* assign, const Workspace& ws,
                                     hipStream_t s) {
  const long total = static_cast<long>(p.n) * (D / 4);
  dim3 grid(static_cast<unsigned>((total + 255) / 256), p.units());
  hipLaunchKernelGGL((broadcast_kernel<D, T>), grid, dim3(256), 0, s, assign, ws.vcb, p.lengths,
                     p.heads, p.n, p.C, static_cast<T*>(p.out));
  return hipGetLastError();
}

hipError_t launch_broadcast(const Problem& p, const int32_t* assign, const Workspace& ws,
                            hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_broadcast_t<32, float>(p, assign, ws, s) : launch_broadcast_t<32, bf16_t>(p, assign, ws, s);
  return p.dtype == 0 ? launch_broadcast_t<64, float>(p, assign, ws, s) : launch_broadcast_t<64, bf16_t>(p, assign, ws, s);
}

template <int D, typename T>
static hipError_t launch_pad_zero_t(const Problem& p, hipStream_t s) {
  const long total = static_cast<long>(p.n) * (D / 4);
  dim3 grid(static_cast<unsigned>((total + 255) / 256), p.units());
  hipLaunchKernelGGL((pad_zero_kernel<D, T>), grid, dim3(256), 0, s, p.lengths, p.heads, p.n,
                     static_cast<T*>(p.out));
  return hipGetLastError();
}

hipError_t launch_pad_zero(const Problem& p, hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_pad_zero_t<32, float>(p, s) : launch_pad_zero_t<32, bf16_t>(p, s);
  return p.dtype == 0 ? launch_pad_zero_t<64, float>(p, s) : launch_pad_zero_t<64, bf16_t>(p, s);
}

template <int D, typename T>
static hipError_t launch_sparse_t(const Problem& p, const Workspace& ws, hipStream_t s) {
  const int kk = p.topk < p.n ? p.topk : p.n;
  const int kpad = ((kk + 15) / 16) * 16;
  const size_t per_wave = static_cast<size_t>(kpad) * ((D + 4) + D) * sizeof(float);
  int wpb = 4;
  while (wpb > 1 && per_wave * wpb > 65536) wpb >>= 1;
  const size_t lds = per_wave * wpb;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&sparse_kernel<D, T>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    attr_set = true;
  }
  const float scale = 1.0f / sqrtf(static_cast<float>(D));
  dim3 grid((p.C + wpb - 1) / wpb, p.units());
  hipLaunchKernelGGL((sparse_kernel<D, T>), grid, dim3(64 * wpb), lds, s,
                     static_cast<const T*>(p.q), static_cast<const T*>(p.k),
                     static_cast<const T*>(p.v), p.lengths, p.heads, p.n, p.C, p.topk, kpad, scale,
                     ws.sizes, ws.offsets, ws.members, ws.topk, ws.mass, ws.vcb,
                     static_cast<T*>(p.out));
  return hipGetLastError();
}

hipError_t launch_sparse(const Problem& p, const Workspace& ws, hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_sparse_t<32, float>(p, ws, s) : launch_sparse_t<32, bf16_t>(p, ws, s);
  return p.dtype == 0 ? launch_sparse_t<64, float>(p, ws, s) : launch_sparse_t<64, bf16_t>(p, ws, s);
}

}  // namespace ca
