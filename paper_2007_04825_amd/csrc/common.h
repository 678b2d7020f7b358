// Device helpers shared by the gfx950 kernels of the clustered-attention library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ca {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef double v4d __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Makes the LDS writes of this wave visible to its other lanes.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Compile-time count for with_count.
template <int M> struct Count {
  static constexpr int value = M;
};

// Calls f(Count<min(n, M)>{}) when n > 0: code that is straight-line over a
// count known at compile time (so that every load in it is unconditional and
// each wait counts exactly the loads still in flight) is instantiated for
// every count from 1 to M and entered for the one that n asks for.
template <int M, class F> __device__ __forceinline__ void with_count(int n, F&& f) {
  if constexpr (M > 0) {
    if (n >= M)
      f(Count<M>{});
    else
      with_count<M - 1>(n, f);
  }
}

// ---------------------------------------------------------------------------
// Element types.  bf16 is carried as raw uint16_t storage.
// ---------------------------------------------------------------------------
struct bf16_t {
  uint16_t x;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x.x) << 16);
}

// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Loads CNT consecutive elements starting at p (aligned to CNT elements) as fp32.
template <int CNT>
__device__ __forceinline__ void load_row(const float* __restrict__ p, float* dst) {
  static_assert(CNT % 4 == 0, "vector width");
#pragma unroll
  for (int i = 0; i < CNT; i += 4) {
    const float4 t = *reinterpret_cast<const float4*>(p + i);
    dst[i] = t.x;
    dst[i + 1] = t.y;
    dst[i + 2] = t.z;
    dst[i + 3] = t.w;
  }
}
template <int CNT>
__device__ __forceinline__ void load_row(const bf16_t* __restrict__ p, float* dst) {
  static_assert(CNT % 4 == 0, "vector width");
#pragma unroll
  for (int i = 0; i < CNT; i += 4) {
    const uint2 t = *reinterpret_cast<const uint2*>(p + i);
    dst[i] = __uint_as_float(t.x << 16);
    dst[i + 1] = __uint_as_float(t.x & 0xffff0000u);
    dst[i + 2] = __uint_as_float(t.y << 16);
    dst[i + 3] = __uint_as_float(t.y & 0xffff0000u);
  }
}

// Stores one fp32 value as the output element type.
__device__ __forceinline__ void store1(float* p, float x) { *p = x; }
__device__ __forceinline__ void store1(bf16_t* p, float x) { p->x = f32_to_bf16_bits(x); }

// Stores 4 consecutive fp32 values (aligned) as the output element type.
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store4(bf16_t* p, float a, float b, float c, float d) {
  uint2 t;
  t.x = static_cast<uint32_t>(f32_to_bf16_bits(a)) | (static_cast<uint32_t>(f32_to_bf16_bits(b)) << 16);
  t.y = static_cast<uint32_t>(f32_to_bf16_bits(c)) | (static_cast<uint32_t>(f32_to_bf16_bits(d)) << 16);
  *reinterpret_cast<uint2*>(p) = t;
}

// ---------------------------------------------------------------------------
// Lengths: lengths[b] clamped to [0, N]; NULL means every row is valid.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int unit_length(const int32_t* __restrict__ lengths, int b, int N) {
  if (lengths == nullptr) return N;
  int n = lengths[b];
  return n < 0 ? 0 : (n > N ? N : n);
}

// ---------------------------------------------------------------------------
// Wave utilities (wave64).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return static_cast<int>(threadIdx.x) & (kWave - 1); }

// Cross-lane moves without the LDS: DPP within 16-lane rows, and the gfx950
// permlane swaps between rows.  The swaps need two distinct registers, so the
// source is first copied explicitly.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf, 0xf, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xf, 0xf, false);
}
__device__ __forceinline__ unsigned vreg_copy(unsigned x) {
  unsigned y;
  asm volatile("v_mov_b32 %0, %1" : "=v"(y) : "v"(x));
  return y;
}
// value of lane (l ^ 32) / (l ^ 16)
__device__ __forceinline__ unsigned lane_xor32_u(unsigned u) {
  const auto p = __builtin_amdgcn_permlane32_swap(u, vreg_copy(u), false, false);
  return (threadIdx.x & 32) ? p[0] : p[1];
}
__device__ __forceinline__ unsigned lane_xor16_u(unsigned u) {
  const auto p = __builtin_amdgcn_permlane16_swap(u, vreg_copy(u), false, false);
  return (threadIdx.x & 16) ? p[0] : p[1];
}
__device__ __forceinline__ float lane_xor32(float x) {
  return __builtin_bit_cast(float, lane_xor32_u(__builtin_bit_cast(unsigned, x)));
}
__device__ __forceinline__ float lane_xor16(float x) {
  return __builtin_bit_cast(float, lane_xor16_u(__builtin_bit_cast(unsigned, x)));
}
__device__ __forceinline__ int lane_xor32(int x) { return static_cast<int>(lane_xor32_u(static_cast<unsigned>(x))); }
__device__ __forceinline__ double lane_xor32(double x) {
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  const uint64_t lo = lane_xor32_u(static_cast<unsigned>(u));
  const uint64_t hi = lane_xor32_u(static_cast<unsigned>(u >> 32));
  return __builtin_bit_cast(double, lo | (hi << 32));
}
__device__ __forceinline__ int lane_xor16(int x) { return static_cast<int>(lane_xor16_u(static_cast<unsigned>(x))); }

// Reductions over the 16 lanes of a row (quad swaps, half-row mirror, row
// mirror); every lane of the row ends with the same value.
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp_f<0xB1>(x));
  x = fmaxf(x, dpp_f<0x4E>(x));
  x = fmaxf(x, dpp_f<0x141>(x));
  return fmaxf(x, dpp_f<0x140>(x));
}
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_f<0xB1>(x);
  x += dpp_f<0x4E>(x);
  x += dpp_f<0x141>(x);
  return x + dpp_f<0x140>(x);
}
// Reductions over lanes c, c+16, c+32, c+48 (one column of an MFMA result).
__device__ __forceinline__ float cross_rows_max(float x) {
  x = fmaxf(x, lane_xor16(x));
  return fmaxf(x, lane_xor32(x));
}
__device__ __forceinline__ float cross_rows_sum(float x) {
  x += lane_xor16(x);
  return x + lane_xor32(x);
}
__device__ __forceinline__ int cross_rows_max(int x) {
  x = max(x, lane_xor16(x));
  return max(x, lane_xor32(x));
}
// Whole-wave reductions; every lane gets the (bitwise identical) result.
__device__ __forceinline__ float wave_max(float x) { return cross_rows_max(row16_max(x)); }
__device__ __forceinline__ float wave_sum(float x) { return cross_rows_sum(row16_sum(x)); }
__device__ __forceinline__ int wave_sum_i(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ int wave_incl_scan(int x) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (l >= o) x += y;
  }
  return x;
}
__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// ---------------------------------------------------------------------------
// MFMA wrappers (gfx950).  For the 16x16 shapes used here:
//   A operand: lane l holds row (l % 16) and k-group (l / 16);
//   B operand: lane l holds column (l % 16) and k-group (l / 16);
//   result   : lane l, register r holds element [4 * (l / 16) + r][l % 16].
// A and B pair their k values by (k-group, position in the register), so any
// permutation of the reduction index applied to both operands is allowed.
// ---------------------------------------------------------------------------
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// bf16 16x16x32: lane l holds row (l % 16) of A and column (l % 16) of B with
// the eight consecutive k of group (l / 16), two bf16 per word in k order
// (the lower k in the low half); the result lane l, register r holds
// [4 (l / 16) + r][l % 16].  Products are exact, sums in fp32.
__device__ __forceinline__ v4f mfma_bf16_16x16x32(v4u a, v4u b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a),
                                                 __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
}
// Exact split of an fp32 value into three bf16 values x = hi + mid + lo by
// truncation (8 + 8 + 8 significant bits); the parts are returned as fp32 bit
// patterns whose low halves are zero.
__device__ __forceinline__ void split3(float x, uint32_t& h, uint32_t& m, uint32_t& l) {
  const uint32_t u = __float_as_uint(x);
  h = u & 0xffff0000u;
  const float r1 = x - __uint_as_float(h);
  m = __float_as_uint(r1) & 0xffff0000u;
  const float r2 = r1 - __uint_as_float(m);
  l = __float_as_uint(r2) & 0xffff0000u;
}
// Eight fp32 values split as above and packed as bf16 operands (k order).
struct Split8 {
  v4u h, m, l;
};
__device__ __forceinline__ Split8 split8(const float* x) {
  Split8 s;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint32_t h0, m0, l0, h1, m1, l1;
    split3(x[2 * e], h0, m0, l0);
    split3(x[2 * e + 1], h1, m1, l1);
    s.h[e] = (h0 >> 16) | h1;
    s.m[e] = (m0 >> 16) | m1;
    s.l[e] = (l0 >> 16) | l1;
  }
  return s;
}
// Eight values that are bf16 values already (widened to fp32), packed.
__device__ __forceinline__ v4u pack_bf16x8(const float* x) {
  v4u p;
#pragma unroll
  for (int e = 0; e < 4; ++e) p[e] = (__float_as_uint(x[2 * e]) >> 16) | (__float_as_uint(x[2 * e + 1]) & 0xffff0000u);
  return p;
}
// A.B with A exact in bf16 and B split: three products, exact up to the fp32
// sums.
__device__ __forceinline__ v4f mfma_split3(v4u a, const Split8& b, v4f c) {
  c = mfma_bf16_16x16x32(a, b.h, c);
  c = mfma_bf16_16x16x32(a, b.m, c);
  c = mfma_bf16_16x16x32(a, b.l, c);
  return c;
}

// A.B with both operands fp32, each split exactly into three bf16 parts
// (x = hi + mid + lo): the six part products of relative size 2^-16 and
// above, smallest first.  The three left out are below 2^-24 |a_k b_k| each,
// so the result matches an fp32 product sum to within a few units of 2^-24
// (products exact, sums in fp32), on the bf16 matrix cores.
__device__ __forceinline__ v4f mfma_split6(const Split8& a, const Split8& b, v4f c) {
  c = mfma_bf16_16x16x32(a.l, b.h, c);
  c = mfma_bf16_16x16x32(a.m, b.m, c);
  c = mfma_bf16_16x16x32(a.h, b.l, c);
  c = mfma_bf16_16x16x32(a.m, b.h, c);
  c = mfma_bf16_16x16x32(a.h, b.m, c);
  c = mfma_bf16_16x16x32(a.h, b.h, c);
  return c;
}
// Softmax weights P in (0, 1] times bf16 values: P keeps its hi and mid parts
// (16 significant bits, each weight short by less than 2^-15 of itself), two
// products; far below the bf16 rounding of the outputs, and the normalisers
// are summed from the unsplit weights.  fp32 values take the six products of
// mfma_split6.
template <typename T>
__device__ __forceinline__ v4f mfma_weights(const float* x8, const Split8& p, v4f c) {
  if constexpr (sizeof(T) == 2) {
    const v4u a = pack_bf16x8(x8);
    c = mfma_bf16_16x16x32(a, p.m, c);
    return mfma_bf16_16x16x32(a, p.h, c);
  } else {
    return mfma_split6(split8(x8), p, c);
  }
}
// Eight values of the element type T (widened to fp32) times a split B on
// the bf16 matrix cores: bf16 values are exact as one operand (three
// products), fp32 values are split as well (six products).
template <typename T>
__device__ __forceinline__ v4f mfma_bf16x(const float* x8, const Split8& b, v4f c) {
  if constexpr (sizeof(T) == 2) {
    return mfma_split3(pack_bf16x8(x8), b, c);
  } else {
    return mfma_split6(split8(x8), b, c);
  }
}

__device__ __forceinline__ v4f mfma_f32_16x16x4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
// fp64 16x16x4: A and B pair as above, but the result of lane l, register r
// is element [l / 16 + 4 * r][l % 16].
__device__ __forceinline__ v4d mfma_f64_16x16x4(double a, double b, v4d c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v4i mfma_i8_16x16x64(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// XCD-aware placement.  The dispatcher hands consecutive workgroups of a
// launch to the eight XCDs in turn, and each XCD has its own L2.  With the
// grid padded to a multiple of eight, workgroup L takes work item
// (L % 8) * (grid / 8) + L / 8, so that consecutive work items (for example
// the tiles of one (batch, head), which read the same keys and values) run on
// one XCD and share its L2.
// ---------------------------------------------------------------------------
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_work_item() {
  const int per = static_cast<int>(gridDim.x) / kXcds;
  const int L = static_cast<int>(blockIdx.x);
  return (L % kXcds) * per + L / kXcds;
}
inline unsigned xcd_grid(long long nwork) {
  return static_cast<unsigned>((nwork + kXcds - 1) / kXcds * kXcds);
}

// ---------------------------------------------------------------------------
// Order-preserving map from fp32 to uint32: a < b  <=>  key(a) < key(b).
// -0 is folded onto +0 so that equal values get equal keys.
// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// Buffer loads: a resource covering [base, base + bytes) turns every load into
// a 32-bit lane offset plus a uniform offset, and reads past the end return 0
// (so tile edges need no guards).
// ---------------------------------------------------------------------------
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), 0x00020000);
}
// Four consecutive elements (fp32 or bf16, 16- or 8-byte aligned) as fp32.
__device__ __forceinline__ void load4(const float* p, float* d) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  d[0] = v.x;
  d[1] = v.y;
  d[2] = v.z;
  d[3] = v.w;
}
__device__ __forceinline__ void load4(const bf16_t* p, float* d) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  d[0] = __uint_as_float(v.x << 16);
  d[1] = __uint_as_float(v.x & 0xffff0000u);
  d[2] = __uint_as_float(v.y << 16);
  d[3] = __uint_as_float(v.y & 0xffff0000u);
}

// CNT consecutive elements (fp32 or bf16) at byte offset voff + soff, as fp32.
template <int CNT>
__device__ __forceinline__ void buf_load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, float* d, float) {
  if constexpr (CNT == 1) {
    d[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
  } else if constexpr (CNT == 2) {
    const auto t = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    d[0] = __uint_as_float(t[0]);
    d[1] = __uint_as_float(t[1]);
  } else {
    static_assert(CNT % 4 == 0, "vector width");
#pragma unroll
    for (int i = 0; i < CNT; i += 4) {
      const auto t = __builtin_amdgcn_raw_buffer_load_b128(r, voff + 4 * i, soff, 0);
      d[i] = __uint_as_float(t[0]);
      d[i + 1] = __uint_as_float(t[1]);
      d[i + 2] = __uint_as_float(t[2]);
      d[i + 3] = __uint_as_float(t[3]);
    }
  }
}
template <int CNT>
__device__ __forceinline__ void buf_load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, float* d, bf16_t) {
  auto two = [&](uint32_t w, float* o) {
    o[0] = __uint_as_float(w << 16);
    o[1] = __uint_as_float(w & 0xffff0000u);
  };
  if constexpr (CNT == 2) {
    two(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0), d);
  } else if constexpr (CNT == 4) {
    const auto t = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    two(t[0], d);
    two(t[1], d + 2);
  } else {
    static_assert(CNT % 8 == 0, "vector width");
#pragma unroll
    for (int i = 0; i < CNT; i += 8) {
      const auto t = __builtin_amdgcn_raw_buffer_load_b128(r, voff + 2 * i, soff, 0);
      two(t[0], d + i);
      two(t[1], d + i + 2);
      two(t[2], d + i + 4);
      two(t[3], d + i + 6);
    }
  }
}

// CNT consecutive fp32 values stored at byte offset voff + soff as the
// element type (bf16: rounded to nearest even); stores past the end are dropped.
template <int CNT>
__device__ __forceinline__ void buf_store(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, const float* s, float) {
  static_assert(CNT % 4 == 0, "vector width");
  typedef unsigned int u4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < CNT; i += 4) {
    const u4 t = {__float_as_uint(s[i]), __float_as_uint(s[i + 1]), __float_as_uint(s[i + 2]), __float_as_uint(s[i + 3])};
    __builtin_amdgcn_raw_buffer_store_b128(t, r, voff + 4 * i, soff, 0);
  }
}
template <int CNT>
__device__ __forceinline__ void buf_store(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, const float* s, bf16_t) {
  static_assert(CNT % 4 == 0, "vector width");
  auto pack = [&](int i) {
    return static_cast<uint32_t>(f32_to_bf16_bits(s[i])) | (static_cast<uint32_t>(f32_to_bf16_bits(s[i + 1])) << 16);
  };
  if constexpr (CNT % 8 == 0) {
    typedef unsigned int u4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int i = 0; i < CNT; i += 8) {
      const u4 t = {pack(i), pack(i + 2), pack(i + 4), pack(i + 6)};
      __builtin_amdgcn_raw_buffer_store_b128(t, r, voff + 2 * i, soff, 0);
    }
  } else {
    typedef unsigned int u2 __attribute__((ext_vector_type(2)));
    const u2 t = {pack(0), pack(2)};
    __builtin_amdgcn_raw_buffer_store_b64(t, r, voff, soff, 0);
  }
}

// Zeroes the arrival counters (sync_ints ints) and both count tables
// (2 tstride words) of unit u of the cooperative K-means with the threads of
// workgroup blk of nblk, in the kernel that runs before it.
__device__ __forceinline__ void coop_reset(int32_t* sync, int sync_ints, uint64_t* tab, int tstride,
                                           int u, int blk, int nblk, int tid, int nthreads) {
  if (blk == 0 && tid < sync_ints) sync[u * sync_ints + tid] = 0;
  uint64_t* t0 = tab + static_cast<size_t>(u) * 2 * tstride;
  for (int x = blk * nthreads + tid; x < 2 * tstride; x += nblk * nthreads) t0[x] = 0ull;
}

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f == 0.0f ? 0.0f : f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace ca
