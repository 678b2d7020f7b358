// Sign-of-random-projection hashing of the queries (Section 3.2.2).
//
// Bit b of the code of query i is [Q_i . P_b > 0].  The projection is
// evaluated in fp64 with fused multiply-adds in the fixed order t = 0..d-1.
// Every product of two fp32 (or bf16) values is exact in fp64, so the sign is
// the sign of the exactly rounded running sum, independent of any reordering
// of the hardware, and agrees with an fp64 evaluation of the definition.
#include "common.h"
#include "kernels.h"

namespace ca {

constexpr int kHashThreads = 256;

template <int D, typename T>
__global__ __launch_bounds__(kHashThreads) void hash_kernel(const T* __restrict__ q,
                                                            const float* __restrict__ planes,
                                                            const int32_t* __restrict__ lengths,
                                                            int heads, int N, int n_bits,
                                                            uint64_t* __restrict__ codes) {
  __shared__ double pl[64 * D];
  const int u = blockIdx.y;
  const int b = u / heads, h = u % heads;
  const int n = unit_length(lengths, b, N);
  const int i = blockIdx.x * kHashThreads + threadIdx.x;
  uint64_t* out = codes + static_cast<size_t>(u) * N;
  if (blockIdx.x * kHashThreads >= n) {  // whole block past the valid length
    if (i < N) out[i] = 0;
    return;
  }
  const float* ph = planes + static_cast<size_t>(h) * n_bits * D;
  for (int x = threadIdx.x; x < n_bits * D; x += kHashThreads) pl[x] = static_cast<double>(ph[x]);
  __syncthreads();
  if (i >= N) return;
  uint64_t code = 0;
  if (i < n) {
    float qf[D];
    load_row<D>(q + (static_cast<size_t>(u) * N + i) * D, qf);
    double qd[D];
#pragma unroll
    for (int t = 0; t < D; ++t) qd[t] = static_cast<double>(qf[t]);
    for (int bb = 0; bb < n_bits; ++bb) {
      const double* w = pl + bb * D;
      double p = 0.0;
#pragma unroll
      for (int t = 0; t < D; ++t) p = fma(qd[t], w[t], p);
      code |= static_cast<uint64_t>(p > 0.0) << bb;
    }
  }
  out[i] = code;
}

// Copies caller-supplied codes, keeping bits below n_bits and zeroing padded rows.
__global__ __launch_bounds__(256) void load_codes_kernel(const uint64_t* __restrict__ in,
                                                         const int32_t* __restrict__ lengths,
                                                         int heads, int N, int n_bits,
                                                         uint64_t* __restrict__ codes) {
  const int u = blockIdx.y;
  const int n = unit_length(lengths, u / heads, N);
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= N) return;
  const uint64_t mask = n_bits >= 64 ? ~0ull : ((1ull << n_bits) - 1);
  const size_t x = static_cast<size_t>(u) * N + i;
  codes[x] = i < n ? (in[x] & mask) : 0ull;
}

template <int D, typename T>
static hipError_t launch_hash_t(const Problem& p, const Workspace& ws, hipStream_t s) {
  dim3 grid((p.n + kHashThreads - 1) / kHashThreads, p.units());
  hipLaunchKernelGGL((hash_kernel<D, T>), grid, dim3(kHashThreads), 0, s,
                     static_cast<const T*>(p.q), p.planes, p.lengths, p.heads, p.n, p.n_bits,
                     ws.codes);
  return hipGetLastError();
}

hipError_t launch_hash(const Problem& p, const Workspace& ws, hipStream_t s) {
  if (p.d == 32) return p.dtype == 0 ? launch_hash_t<32, float>(p, ws, s) : launch_hash_t<32, bf16_t>(p, ws, s);
  return p.dtype == 0 ? launch_hash_t<64, float>(p, ws, s) : launch_hash_t<64, bf16_t>(p, ws, s);
}

hipError_t launch_load_codes(const Problem& p, const uint64_t* codes_in, const Workspace& ws,
                             hipStream_t s) {
  dim3 grid((p.n + 255) / 256, p.units());
  hipLaunchKernelGGL(load_codes_kernel, grid, dim3(256), 0, s, codes_in, p.lengths, p.heads, p.n,
                     p.n_bits, ws.codes);
  return hipGetLastError();
}

}  // namespace ca
