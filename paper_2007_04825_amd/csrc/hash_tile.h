// Sign-of-random-projection hashing of one 16-query tile (Section 3.2.2) on
// the bf16 matrix cores, exact with respect to the fp64 definition.
//
// Bit b of the code of query i is [Q_i . P_b > 0], where the projection is the
// fp64 sum over t = 0..d-1 in that order (each product of two fp32 values is
// exact in fp64, so the sum is that of a sequential fma chain).
//
// Fast path.  The planes are bf16 values (the hash draws them that way), and an
// fp32 query value splits exactly into three bf16 parts x = hi + mid + lo
// (truncation: 8 + 8 + 8 significant bits); a bf16 query value is its own hi
// part.  v_mfma_f32_16x16x32_bf16 forms the products exactly and accumulates
// them in fp32, so the result S of m = 3d (fp32) or m = d (bf16) exact terms
// obeys, with unit roundoff u = 2^-24 (2^-23 if the accumulation truncated),
//     |S - Q . P| <= m u (1 + 2^-7) sum_t |Q_t P_t| <= m u (1 + 2^-7) |Q| |P|
// by Cauchy-Schwarz: at most 2^-16.4 |Q| |P| (fp32, d <= 64; 2^-15.4 under
// truncation) and 2^-18 |Q| |P| (bf16; 2^-17 under truncation).  Parts and
// products below the fp32 normal range, flushed to zero, change S by less
// than 2^-120 |P|, negligible once |Q|^2 >= 2^-45 (checked).  Every sign with
// |S| above the band, 2^-14 |Q| |P| (fp32) or 2^-16 |Q| |P| (bf16), is
// therefore the exact sign; the projections inside it (about 4e-4 and 1e-4 of
// them for Gaussian data) are recomputed by their lane as the sequential fp64
// fma chain, which reproduces the definition bit for bit.  Norms too small or
// too large for the fp32 test send the projection to the fp64 chain as well.
//
// Planes that are not bf16 values make every projection take the fp64 chain
// (correct, slower).
//
// Operand layouts (16x16x32 bf16): lane l holds row (l % 16) and the eight
// consecutive k of group (l / 16); the result lane l, register r holds
// [4 (l / 16) + r][l % 16].  Rows are planes, columns queries, so that a lane
// ends with sixteen signs of one query (planes 16 pt + 4 (l / 16) + r) and
// four lanes together hold its whole code.
#pragma once
#include "common.h"

namespace ca {


// A operands of the 64 plane rows (four 16-plane tiles) for D/32 k-chunks;
// thr: |P_b|^2 for b = 0..63 in LDS (read per tile, so that the
// sixteen values a lane needs do not occupy registers across the tile loop);
// valid: for the planes whose signs this lane receives (16 pt + 4 (lane /
// 16) + r), whether they exist (bit 4 pt + r).
template <int D>
struct PlaneOps {
  v4u b[D / 32][4];
  const float* thr;
  uint32_t valid;
  bool norms_ok;  // every plane norm within the range of the fp32 test
};

// Floats per staged plane row: a stride of 4 mod 64 puts the rows that the
// sixteen lanes of a lane group read together in distinct LDS banks.
template <int D>
constexpr int kPlaneRow = D + 4;

// The n_bits planes of one head [n_bits][D] are copied into
// sp[64][kPlaneRow<D>] (LDS; rows past n_bits are zero) by the NT threads of
// the workgroup, so that the waves read their operands from LDS instead of
// all fetching the same few kilobytes from L2.  The copy is split in two:
// fetch_planes requests this thread's part, store_planes writes it to LDS.
// Loads issued in between (the first query tile) stay in flight while the
// stores wait for the planes alone.  The caller synchronises the workgroup
// before sp is read.
template <int D, int NT>
struct PlaneStage {
  static constexpr int kPer = (64 * D / 4 + NT - 1) / NT;  // float4 per thread
  float4 v[kPer];
};
template <int D, int NT>
__device__ __forceinline__ void fetch_planes(const float* __restrict__ ph, int n_bits,
                                             PlaneStage<D, NT>& st, int tid) {
  // through a buffer resource: every load is issued without a branch (so
  // that the compiler counts them), positions past the planes reading 0
  const __amdgpu_buffer_rsrc_t rp = make_rsrc(ph, static_cast<uint32_t>(n_bits) * D * 4);
#pragma unroll
  for (int i = 0; i < PlaneStage<D, NT>::kPer; ++i) {
    const int x = tid + i * NT;
    const auto t = __builtin_amdgcn_raw_buffer_load_b128(rp, static_cast<uint32_t>(x) * 16, 0, 0);
    st.v[i] = make_float4(__uint_as_float(t[0]), __uint_as_float(t[1]), __uint_as_float(t[2]), __uint_as_float(t[3]));
  }
}
template <int D, int NT>
__device__ __forceinline__ void store_planes(const PlaneStage<D, NT>& st, float* sp, int tid) {
  // with NT * kPer = 64 D / 4 every thread stores all of its parts (no branch
  // for the compiler to sink the loads into)
  constexpr bool kExact = NT * PlaneStage<D, NT>::kPer == 64 * D / 4;
#pragma unroll
  for (int i = 0; i < PlaneStage<D, NT>::kPer; ++i) {
    const int x = tid + i * NT;
    if (kExact || x < 64 * D / 4) {
      const int row = x / (D / 4), col = 4 * (x % (D / 4));
      *reinterpret_cast<float4*>(sp + row * kPlaneRow<D> + col) = st.v[i];
    }
  }
}

// Builds this lane's plane operands from the staged planes sp[64][kPlaneRow<D>].  The
// lanes of a wave read every plane value between them; returns true (in every
// lane) if one of them is not a bf16 value.  thr: 64 floats of LDS private to
// the wave, which receive the plane thresholds.
template <int D>
__device__ __forceinline__ bool load_plane_ops(const float* sp, int n_bits, int lane, PlaneOps<D>& P,
                                               float* thr) {
  const int c = lane & 15, g = lane >> 4;
  uint32_t low = 0;
  float sq[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kc = 0; kc < D / 32; ++kc)
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) {
      const int plane = pt * 16 + c;
      v4u w = {0u, 0u, 0u, 0u};
      if (plane < n_bits) {
        const float* pr = sp + plane * kPlaneRow<D> + kc * 32 + 8 * g;
        const float4 x0 = *reinterpret_cast<const float4*>(pr);
        const float4 x1 = *reinterpret_cast<const float4*>(pr + 4);
        const uint32_t u[8] = {__float_as_uint(x0.x), __float_as_uint(x0.y), __float_as_uint(x0.z),
                               __float_as_uint(x0.w), __float_as_uint(x1.x), __float_as_uint(x1.y),
                               __float_as_uint(x1.z), __float_as_uint(x1.w)};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          low |= u[e] & 0xffffu;
          sq[pt] = fmaf(__uint_as_float(u[e]), __uint_as_float(u[e]), sq[pt]);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = (u[2 * e] >> 16) | (u[2 * e + 1] & 0xffff0000u);
      }
      P.b[kc][pt] = w;
    }
  bool ok = true;
  P.valid = 0u;
#pragma unroll
  for (int pt = 0; pt < 4; ++pt) {
    const float n2 = cross_rows_sum(sq[pt]);  // |P|^2 of plane 16 pt + lane % 16
    if (pt * 16 + c < n_bits) ok = ok && n2 >= 0x1p-45f && n2 < 0x1p+50f;
    if (g == 0) thr[pt * 16 + c] = n2;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (pt * 16 + 4 * g + r < n_bits) P.valid |= 1u << (4 * pt + r);
  }
  wave_lds_sync();
  P.thr = thr;
  P.norms_ok = __ballot(!ok) == 0ull;
  return __ballot(low != 0u) != 0ull;
}

// The projection as defined: fp64 fma chain over t = 0..D-1.  The operands
// are fetched sixteen dimensions at a time, all loads of a group in flight
// together.
template <int D, typename T>
__device__ __forceinline__ double exact_projection(const T* __restrict__ qr, const float* pr) {
  double p = 0.0;
#pragma unroll 1
  for (int t0 = 0; t0 < D; t0 += 16) {
    float x[16], y[16];
    load_row<16>(qr + t0, x);
    load_row<16>(pr + t0, y);
#pragma unroll
    for (int t = 0; t < 16; ++t) p = fma(static_cast<double>(x[t]), static_cast<double>(y[t]), p);
  }
  return p;
}

// Raw query values of one tile as this lane loads them: row row0 + lane % 16,
// dimensions kc * 32 + 8 (lane / 16) .. + 7 for each k-chunk kc (the next tile
// is requested while the current one is on the matrix cores).  The loads go
// through a buffer resource over the nq valid rows: every load is issued
// without a branch (so that the compiler counts the loads in flight), and
// rows past nq read 0.
template <int D, typename T>
struct TileRaw {
  uint4 w[D / 32][sizeof(T) / 2];  // 8 values: two uint4 of fp32, or one of bf16
};
template <int D, typename T>
__device__ __forceinline__ TileRaw<D, T> load_tile(const T* __restrict__ qu, int row0, int nq,
                                                   int lane) {
  const int c = lane & 15, g = lane >> 4;
  constexpr uint32_t ESZ = sizeof(T);
  const __amdgpu_buffer_rsrc_t rq =
      make_rsrc(qu + static_cast<size_t>(nq > 0 ? row0 : 0) * D, static_cast<uint32_t>(nq > 0 ? nq : 0) * D * ESZ);
  TileRaw<D, T> r;
#pragma unroll
  for (int kc = 0; kc < D / 32; ++kc)
#pragma unroll
    for (int h = 0; h < static_cast<int>(ESZ) / 2; ++h) {
      const uint32_t voff = (static_cast<uint32_t>(c) * D + 8 * g + 32 * kc) * ESZ + 16 * h;
      const auto t = __builtin_amdgcn_raw_buffer_load_b128(rq, voff, 0, 0);
      r.w[kc][h] = make_uint4(t[0], t[1], t[2], t[3]);
    }
  return r;
}

// Writes this lane's part of a loaded tile to stash[16][kPlaneRow<D>] as fp32
// (row lane % 16), so that the exact fallback reads the query rows from LDS
// instead of fetching them again from HBM.
template <int D, typename T>
__device__ __forceinline__ void stash_tile(const TileRaw<D, T>& raw, float* stash, int lane) {
  const int c = lane & 15, g = lane >> 4;
#pragma unroll
  for (int kc = 0; kc < D / 32; ++kc) {
    float* dst = stash + c * kPlaneRow<D> + kc * 32 + 8 * g;
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<uint4*>(dst) = raw.w[kc][0];
      *reinterpret_cast<uint4*>(dst + 4) = raw.w[kc][1];
    } else {
      const uint4 w = raw.w[kc][0];
      *reinterpret_cast<float4*>(dst) = make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                                                    __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u));
      *reinterpret_cast<float4*>(dst + 4) = make_float4(__uint_as_float(w.z << 16), __uint_as_float(w.z & 0xffff0000u),
                                                        __uint_as_float(w.w << 16), __uint_as_float(w.w & 0xffff0000u));
    }
  }
}

// Query operands of one k-chunk: hi / mid / lo parts, and the sum of squares
// of the eight values.
struct QueryOps {
  v4u hi, mid, lo;
  float sq;
};
__device__ __forceinline__ QueryOps query_ops(const uint4 (&w)[2]) {
  const float x[8] = {__uint_as_float(w[0].x), __uint_as_float(w[0].y), __uint_as_float(w[0].z),
                      __uint_as_float(w[0].w), __uint_as_float(w[1].x), __uint_as_float(w[1].y),
                      __uint_as_float(w[1].z), __uint_as_float(w[1].w)};
  QueryOps o;
  o.sq = 0.0f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint32_t h0, m0, l0, h1, m1, l1;
    split3(x[2 * e], h0, m0, l0);
    split3(x[2 * e + 1], h1, m1, l1);
    o.hi[e] = (h0 >> 16) | h1;
    o.mid[e] = (m0 >> 16) | m1;
    o.lo[e] = (l0 >> 16) | l1;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) o.sq = fmaf(x[e], x[e], o.sq);
  return o;
}
__device__ __forceinline__ QueryOps query_ops(const uint4 (&w)[1]) {
  QueryOps o;
  o.hi = v4u{w[0].x, w[0].y, w[0].z, w[0].w};
  o.mid = o.lo = v4u{0u, 0u, 0u, 0u};
  o.sq = 0.0f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float a = __uint_as_float(o.hi[e] << 16), b = __uint_as_float(o.hi[e] & 0xffff0000u);
    o.sq = fmaf(a, a, fmaf(b, b, o.sq));
  }
  return o;
}

// Code of query row0 + (lane % 16) (every lane of that column returns it).
// qu: the unit's query rows; raw: this tile as loaded by load_tile; nq: valid
// rows from row0 (>= 1); sp: the staged planes; exact_all: planes are not
// bf16 values; stash: 16 kPlaneRow<D> floats of LDS private to the wave, or
// null (the fallback then reads the query rows from qu).
template <int D, typename T>
__device__ uint64_t hash_tile(const T* __restrict__ qu, const TileRaw<D, T>& raw, int row0, int nq,
                              const float* sp, int n_bits, const PlaneOps<D>& P,
                              bool exact_all, int lane, float* stash) {
  const int c = lane & 15, g = lane >> 4;
  v4f s[4];
#pragma unroll
  for (int pt = 0; pt < 4; ++pt) s[pt] = v4f{0.f, 0.f, 0.f, 0.f};
  float qsq = 0.0f;
  if (!exact_all) {
#pragma unroll
    for (int kc = 0; kc < D / 32; ++kc) {
      const QueryOps o = query_ops(raw.w[kc]);
      qsq += o.sq;
#pragma unroll
      for (int pt = 0; pt < 4; ++pt) {
        s[pt] = mfma_bf16_16x16x32(P.b[kc][pt], o.hi, s[pt]);
        if constexpr (sizeof(T) == 4) {
          s[pt] = mfma_bf16_16x16x32(P.b[kc][pt], o.mid, s[pt]);
          s[pt] = mfma_bf16_16x16x32(P.b[kc][pt], o.lo, s[pt]);
        }
      }
    }
  }
  qsq = cross_rows_sum(qsq);  // |Q|^2 of query c in all four lanes of column c
  // the square of the band's relative width (a power of two: exact)
  constexpr float kBand2 = sizeof(T) == 4 ? 0x1p-28f : 0x1p-32f;
  const float qband = kBand2 * qsq;
  // signs and certainties as lane bit masks, bit 4 pt + r = plane 16 pt + 4 g + r
  v4f thr[4];
#pragma unroll
  for (int pt = 0; pt < 4; ++pt) thr[pt] = *reinterpret_cast<const v4f*>(P.thr + 16 * pt + 4 * g);
  uint32_t pos = 0u, sure = 0u;
#pragma unroll
  for (int k = 15; k >= 0; --k) {
    const float sv = s[k >> 2][k & 3];
    pos = (pos << 1) | (sv > 0.0f ? 1u : 0u);
    sure = (sure << 1) | (sv * sv > qband * thr[k >> 2][k & 3] ? 1u : 0u);
  }
  const uint32_t valid = c < nq ? P.valid : 0u;
  const bool fast = !exact_all && P.norms_ok && qsq >= 0x1p-45f && qsq < 0x1p+50f;
  const uint32_t unc = fast ? (valid & ~sure) : valid;
  pos &= valid;
  // projections inside the band: the fp64 chain (rare, divergent)
  if (__ballot(unc != 0u) != 0ull) {
    if (stash != nullptr) {
      stash_tile<D, T>(raw, stash, lane);
      wave_lds_sync();
    }
    uint32_t m = unc;
    while (m != 0u) {
      const int k = __ffs(m) - 1;
      m &= m - 1;
      const float* pr = sp + ((k >> 2) * 16 + 4 * g + (k & 3)) * kPlaneRow<D>;
      const double p = stash != nullptr
                           ? exact_projection<D, float>(stash + c * kPlaneRow<D>, pr)
                           : exact_projection<D, T>(qu + static_cast<size_t>(row0 + c) * D, pr);
      pos = p > 0.0 ? (pos | (1u << k)) : (pos & ~(1u << k));
    }
    if (stash != nullptr) wave_lds_sync();  // read before the next tile's stash
  }
  // this lane's 16 bits in place, then OR over the four lanes of the column
  uint32_t lo = ((pos & 0xfu) | ((pos & 0xf0u) << 12)) << (4 * g);
  uint32_t hi = (((pos >> 8) & 0xfu) | (((pos >> 12) & 0xfu) << 16)) << (4 * g);
  lo |= lane_xor16_u(lo);
  hi |= lane_xor16_u(hi);
  lo |= lane_xor32_u(lo);
  hi |= lane_xor32_u(hi);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

}  // namespace ca
