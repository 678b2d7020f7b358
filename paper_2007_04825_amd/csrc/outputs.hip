// Output stages used when the centroid-attention kernel does not write the
// rows itself (sequences longer than one key chunk) and for padding.
//
// broadcast_kernel (clustered, Eq. 6): every valid query row receives V^c of
//   its cluster; padded rows receive 0.  Four float4 parts of rows per
//   thread, 256 parts apart, so that every store instruction is fully
//   coalesced (a quarter of the workgroups of one part per thread: sweep
//   point 16.3 -> 14.6 us).
// pad_zero_kernel: rows past a sequence's length receive 0.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace ca {

template <int D, typename T>
__global__ __launch_bounds__(256) void broadcast_kernel(const int32_t* __restrict__ assign,
                                                        const float* __restrict__ vc,
                                                        const int32_t* __restrict__ lengths,
                                                        int heads, int N, int C,
                                                        T* __restrict__ out) {
  constexpr int PR = D / 4;  // float4 parts per row
  constexpr int PER = 4;     // parts per thread, 256 apart
  const int u = blockIdx.y;
  const int n = unit_length(lengths, u / heads, N);
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int idx = (blockIdx.x * PER + k) * 256 + threadIdx.x;
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

// ---------------------------------------------------------------------------
// Host launchers.
// ---------------------------------------------------------------------------
template <int D, typename T>
static hipError_t launch_broadcast_t(const Problem& p, const int32_t* assign, const Workspace& ws,
                                     hipStream_t s) {
  const long total = static_cast<long>(p.n) * (D / 4);
  dim3 grid(static_cast<unsigned>((total + 4 * 256 - 1) / (4 * 256)), p.units());
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

}  // namespace ca
