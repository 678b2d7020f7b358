// Sign-of-random-projection hashing of the queries (Section 3.2.2) for the
// long-sequence path; short sequences are hashed inside the clustering kernel.
// The arithmetic (bf16 matrix cores with an exact fp64 fallback inside the
// rounding band) is described in hash_tile.h.
#include "common.h"
#include "hash_tile.h"
#include "kernels.h"

namespace ca {

constexpr int kHashThreads = 256;
constexpr int kHashQB = 256;  // queries per workgroup: four 16-query tiles per wave

// Rows past the valid length get code 0 and, when out is given, a zero output
// row.  The workgroups of each unit also zero the unit's arrival counters and
// first count table of the cooperative K-means, which runs next.
// Four waves per SIMD (at most 128 registers): the hashing is bound by
// instruction issue, and a fourth wave per SIMD keeps all of the grid resident
// (measured 35 -> 32 us at N = 32768 fp32, 45 -> 40 us at N = 65536 bf16).
template <int D, typename T>
__global__ __launch_bounds__(kHashThreads) __attribute__((amdgpu_waves_per_eu(4))) void hash_kernel(const T* __restrict__ q,
                                                            const float* __restrict__ planes,
                                                            const int32_t* __restrict__ lengths,
                                                            int heads, int N, int n_bits,
                                                            uint64_t* __restrict__ codes,
                                                            T* __restrict__ out,
                                                            int32_t* __restrict__ sync,
                                                            uint64_t* __restrict__ ctab, int tstride) {
  const int u = blockIdx.y;
  coop_reset(sync, kSyncInts, ctab, tstride, u, blockIdx.x, gridDim.x, threadIdx.x, kHashThreads);
  const int b = u / heads, h = u % heads;
  const int n = unit_length(lengths, b, N);
  const int q0 = blockIdx.x * kHashQB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
  if (nq <= 0) return;  // uniform over the workgroup
  __shared__ __align__(16) float sp[64 * kPlaneRow<D>];
  __shared__ __align__(16) float stash[kHashThreads / 64][16 * kPlaneRow<D>];  // per-wave query tile
  __shared__ __align__(16) float sthr[kHashThreads / 64][64];                   // per-wave plane thresholds
  const float* ph = planes + static_cast<size_t>(h) * n_bits * D;
  const T* qu = q + static_cast<size_t>(u) * N * D;
  const int ntile = (nq + 15) / 16;
  constexpr int kStep = kHashThreads / 64;
  // planes requested, then the first query tile, which stays in flight while
  // the planes go to LDS
  // (the scheduling barriers keep that order of the loads)
  PlaneStage<D, kHashThreads> stage;
  fetch_planes<D, kHashThreads>(ph, n_bits, stage, tid);
  __builtin_amdgcn_sched_barrier(0);
  const int wu = __builtin_amdgcn_readfirstlane(wave);  // uniform: the tile's buffer resource in scalars
  TileRaw<D, T> nxt = load_tile<D, T>(qu, q0 + wu * 16, wu < ntile ? min(16, n - q0 - wu * 16) : 0, lane);
  __builtin_amdgcn_sched_barrier(0);
  store_planes<D, kHashThreads>(stage, sp, tid);
  __syncthreads();
  PlaneOps<D> P;
  const bool exact_all = load_plane_ops<D>(sp, n_bits, lane, P, sthr[wave]);
  for (int tile = wu; tile < ntile; tile += kStep) {
    const int r0 = q0 + tile * 16;
    const TileRaw<D, T> cur = nxt;
    const int t2 = tile + kStep;
    // issued in every iteration (past the last tile it reads nothing), so that
    // the wait for this tile does not take the next one's loads with it
    nxt = load_tile<D, T>(qu, q0 + t2 * 16, t2 < ntile ? min(16, n - q0 - t2 * 16) : 0, lane);
    const uint64_t code = hash_tile<D, T>(qu, cur, r0, min(16, n - r0), sp, n_bits, P, exact_all, lane, stash[wave]);
    if (lane < 16 && r0 + lane < n) cu[r0 + lane] = code;
  }
}

// Copies caller-supplied codes, keeping bits below n_bits and zeroing padded
// rows; zeroes the cooperative K-means' counters and table as hash_kernel does.
__global__ __launch_bounds__(256) void load_codes_kernel(const uint64_t* __restrict__ in,
                                                         const int32_t* __restrict__ lengths,
                                                         int heads, int N, int n_bits,
                                                         uint64_t* __restrict__ codes,
                                                         int32_t* __restrict__ sync,
                                                         uint64_t* __restrict__ ctab, int tstride) {
  const int u = blockIdx.y;
  coop_reset(sync, kSyncInts, ctab, tstride, u, blockIdx.x, gridDim.x, threadIdx.x, 256);
  const int n = unit_length(lengths, u / heads, N);
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= N) return;
  const uint64_t mask = n_bits >= 64 ? ~0ull : ((1ull << n_bits) - 1);
  const size_t x = static_cast<size_t>(u) * N + i;
  codes[x] = i < n ? (in[x] & mask) : 0ull;
}

// Hyperplanes drawn on the device when the caller gives none (Section 3.2.2
// draws them at random).  Thread t makes entries 4t .. 4t + 3 of the flat
// planes[heads][n_bits][d] from one block of the counter-based generator
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011), counter (t, 0, 0, 0)
// and key (seed, 0): its words (0, 1) and (2, 3) are two pairs of uniforms
// u1 = ((w >> 11) + 1) 2^-53 in (0, 1], u2 = (w >> 11) 2^-53 in [0, 1), and
// the Box-Muller transform (Box and Muller 1958) turns a pair into the two
// standard normal deviates sqrt(-2 ln u1) (cos, sin)(2 pi u2), evaluated in
// fp64 and stored as fp32.
constexpr uint64_t kPhiloxMul0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kPhiloxMul1 = 0xCA5A826395121157ull;
constexpr uint64_t kPhiloxInc0 = 0x9E3779B97F4A7C15ull;  // key increments between rounds
constexpr uint64_t kPhiloxInc1 = 0xBB67AE8584CAA73Bull;

__global__ __launch_bounds__(256) void planes_kernel(uint64_t seed, int count,
                                                     float* __restrict__ planes) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (4 * static_cast<long long>(t) >= count) return;
  uint64_t w0 = static_cast<uint64_t>(t), w1 = 0, w2 = 0, w3 = 0;
  uint64_t ka = seed, kb = 0;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint64_t hi0 = __umul64hi(kPhiloxMul0, w0), lo0 = kPhiloxMul0 * w0;
    const uint64_t hi1 = __umul64hi(kPhiloxMul1, w2), lo1 = kPhiloxMul1 * w2;
    w0 = hi1 ^ w1 ^ ka;
    w1 = lo1;
    w2 = hi0 ^ w3 ^ kb;
    w3 = lo0;
    ka += kPhiloxInc0;
    kb += kPhiloxInc1;
  }
  const uint64_t words[4] = {w0, w1, w2, w3};
#pragma unroll
  for (int pair = 0; pair < 2; ++pair) {
    const double u1 = static_cast<double>((words[2 * pair] >> 11) + 1) * 0x1.0p-53;
    const double u2 = static_cast<double>(words[2 * pair + 1] >> 11) * 0x1.0p-53;
    const double r = sqrt(-2.0 * log(u1));
    const double angle = 6.283185307179586476925286766559 * u2;
    const int i = 4 * t + 2 * pair;
    if (i < count) planes[i] = static_cast<float>(r * cos(angle));
    if (i + 1 < count) planes[i + 1] = static_cast<float>(r * sin(angle));
  }
}

hipError_t launch_planes(const Problem& p, uint64_t seed, float* planes, hipStream_t s) {
  const int count = p.heads * p.n_bits * p.d;
  const int threads = (count + 3) / 4;
  hipLaunchKernelGGL(planes_kernel, dim3((threads + 255) / 256), dim3(256), 0, s, seed, count, planes);
  return hipGetLastError();
}

template <int D, typename T>
static hipError_t launch_hash_t(const Problem& p, const Workspace& ws, hipStream_t s) {
  dim3 grid((p.n + kHashQB - 1) / kHashQB, p.units());
  hipLaunchKernelGGL((hash_kernel<D, T>), grid, dim3(kHashThreads), 0, s,
                     static_cast<const T*>(p.q), p.planes, p.lengths, p.heads, p.n, p.n_bits,
                     ws.codes, p.lengths ? static_cast<T*>(p.out) : nullptr, ws.sync, ws.ctab,
                     coop_table_stride(p.C));
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
                     p.n_bits, ws.codes, ws.sync, ws.ctab, coop_table_stride(p.C));
  return hipGetLastError();
}

}  // namespace ca
