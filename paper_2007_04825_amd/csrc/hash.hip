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
constexpr int kHashQB = 256;  // queries per workgroup: four 16-query tiles per wave

// Projections on the fp64 matrix cores: v_mfma_f64_16x16x4f64 with 16
// queries as rows and 16 planes as columns, four plane tiles for the 64 bit
// positions.  The reduction index t runs as t = 4s + g (K-step s, lane group
// g); the instruction adds its four products in that order with one rounding
// each, exactly like a sequential fma chain over t = 0..d-1, which is the
// order the projections are defined with.  The result lane layout is row
// g + 4r (register r), column lane % 16, so one wave ballot per (plane tile,
// register) yields 16 plane bits for each of four queries.  The planes stay
// in registers while a wave hashes its four query tiles.  Rows past the valid
// length get code 0 and, when out is given, a zero output row.
template <int D, typename T>
__global__ __launch_bounds__(kHashThreads) void hash_kernel(const T* __restrict__ q,
                                                            const float* __restrict__ planes,
                                                            const int32_t* __restrict__ lengths,
                                                            int heads, int N, int n_bits,
                                                            uint64_t* __restrict__ codes,
                                                            T* __restrict__ out) {
  constexpr int KS = D / 4;
  const int u = blockIdx.y;
  const int b = u / heads, h = u % heads;
  const int n = unit_length(lengths, b, N);
  const int q0 = blockIdx.x * kHashQB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, g = lane >> 4;
  uint64_t* cu = codes + static_cast<size_t>(u) * N;
  for (int x = tid; x < kHashQB; x += kHashThreads) {
    const int i = q0 + x;
    if (i < N && i >= n) cu[i] = 0;
  }
  if (out != nullptr) {
    for (int x = tid; x < kHashQB * (D / 4); x += kHashThreads) {
      const int i = q0 + x / (D / 4);
      if (i < N && i >= n)
        store4(out + (static_cast<size_t>(u) * N + i) * D + (x % (D / 4)) * 4, 0.f, 0.f, 0.f, 0.f);
    }
  }
  const int nq = min(kHashQB, n - q0);
  const int ntile = (nq + 15) / 16;  // <= 16 tiles; wave w hashes tiles w, w+4, w+8, w+12
  if (wave >= ntile) return;         // no workgroup barrier follows
  double bp[4][KS];
#pragma unroll
  for (int pt = 0; pt < 4; ++pt) {
    const int plane = pt * 16 + c;
    const float* pr = planes + (static_cast<size_t>(h) * n_bits + min(plane, n_bits - 1)) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) bp[pt][s] = plane < n_bits ? static_cast<double>(pr[4 * s + g]) : 0.0;
  }
  const int my_r = lane >> 2, my_g = lane & 3;
  // query operand of a tile: dims 4s + g of row tile * 16 + c (the next tile
  // is requested while the current one is on the matrix cores)
  auto fetch = [&](int tile, float* dst) {
    const int row = tile * 16 + c;
    const T* qr = q + (static_cast<size_t>(u) * N + q0 + (row < nq ? row : 0)) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s) dst[s] = row < nq ? to_f32(qr[4 * s + g]) : 0.0f;
  };
  float nxt[KS];
  fetch(wave, nxt);
  for (int tile = wave; tile < ntile; tile += 4) {
    const int qw = tile * 16;
    double a[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) a[s] = static_cast<double>(nxt[s]);
    if (tile + 4 < ntile) fetch(tile + 4, nxt);
    v4d acc[4];
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) acc[pt] = v4d{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int pt = 0; pt < 4; ++pt) acc[pt] = mfma_f64_16x16x4(a[s], bp[pt][s], acc[pt]);
    // query g' + 4r of the tile sits in register r of lane group g'
    uint64_t code = 0;
#pragma unroll
    for (int pt = 0; pt < 4; ++pt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint64_t bl = __ballot(acc[pt][r] > 0.0);
        if (r == my_r) code |= ((bl >> (16 * my_g)) & 0xffffull) << (16 * pt);
      }
    if (lane < 16 && qw + lane < nq) cu[q0 + qw + lane] = code;
  }
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
  dim3 grid((p.n + kHashQB - 1) / kHashQB, p.units());
  hipLaunchKernelGGL((hash_kernel<D, T>), grid, dim3(kHashThreads), 0, s,
                     static_cast<const T*>(p.q), p.planes, p.lengths, p.heads, p.n, p.n_bits,
                     ws.codes, p.lengths ? static_cast<T*>(p.out) : nullptr);
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
