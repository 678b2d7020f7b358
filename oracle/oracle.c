/*
 * Plain fp64 CPU oracle for clustered and improved-clustered attention
 * (Vyas, Katharopoulos, Fleuret: "Fast Transformers with Clustered Attention").
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the independent reference that the
 * GPU library is checked against.  Nothing in the product path may link, load
 * or call it; only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header, table or constant with the GPU
 * library.
 *
 * Every function below follows one step of the paper, named in its comment by
 * section and equation.  Arithmetic is IEEE fp64 on the exact input values
 * (fp32 and bf16 inputs widen to fp64 without rounding).  Loops run in the
 * plain order the definition suggests; there is no blocking or fusion.
 *
 * Readings of points the paper leaves open (each one is listed with its reason
 * in the design notes of the repository):
 *   - hash bit b of query i is [Q_i . P_b > 0]; an exact zero gives 0; bit b is
 *     plane b, least significant first; bits >= n_bits are 0.
 *   - K-means runs in Hamming space with binary centroids; the update is the
 *     per-bit majority of the members (a tie gives 0); an empty cluster keeps
 *     its previous centroid; the assignment tie goes to the smaller cluster
 *     index; initial centroids are the codes of queries floor(j*n/C_eff).
 *   - "L Lloyd iterations" = L rounds of (assign, update); the partition S is
 *     the assignment of the L-th round.
 *   - logits carry the 1/sqrt(D_k) factor everywhere, also in Eq. 11.
 *   - keys and queries at positions >= n (the valid length) are masked out;
 *     C_eff = min(C, n), k_eff = min(k, n).
 *   - the top-k set ranks keys by their centroid logit (equivalently by A^c,
 *     softmax being monotone); a tie goes to the smaller key index.
 *   - oracle-top (the paper's comparison variant that keeps each query's k
 *     keys of highest attention): the weights are the softmax renormalised
 *     over those k keys; the ranking and its ties follow the top-k rule above.
 *   - gradients (the paper trains through the operator but writes no
 *     backward pass): the partition and the top-k sets are discrete and held
 *     constant; the gradient flows through the centroids (Eq. 3), the
 *     centroid softmax (Eq. 4-5), the broadcast (Eq. 6) and, for the improved
 *     variant, through the exact top-k logits, the mass m_j and the rest
 *     part Vb_j, all of which depend on the centroid attention.
 *
 * Parity status: every function here is pinned by the CPU test-suite against
 * something other than itself (exact rational arithmetic, brute force,
 * closed forms, special cases that reduce to textbook attention, finite
 * differences); none is marked unpinned.  The projections are pinned to
 * exact rational dot products within the fp64 summation bound and to the
 * hash codes; exact attention to numpy's softmax attention, closed forms and
 * its permutation symmetries; the seeded planes' generator to numpy's own
 * Philox4x64-10 word for word, and their deviates to the Box-Muller polar
 * identities and the normal distribution.  The whole file also runs clean under
 * AddressSanitizer and UndefinedBehaviorSanitizer (sanitize_check.c).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <omp.h>

#include "oracle.h"

/* ------------------------------------------------------------------------ */
/* Section 3.1, Eq. (1)-(2): exact softmax attention of one (batch, head).     */
/* out_i = sum_l softmax_l(Q_i . K_l / sqrt(d)) V_l over the n valid keys.     */
/* ------------------------------------------------------------------------ */
void orc_full_attention(const double* q, const double* k, const double* v,
                        int64_t n, int d, double* out) {
  const double scale = 1.0 / sqrt((double)d);
  double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  for (int64_t i = 0; i < n; ++i) {
    double m = -INFINITY;
    for (int64_t l = 0; l < n; ++l) {
      double dot = 0.0;
      for (int t = 0; t < d; ++t) dot += q[i * d + t] * k[l * d + t];
      s[l] = dot * scale;
      if (s[l] > m) m = s[l];
    }
    double z = 0.0;
    for (int64_t l = 0; l < n; ++l) {
      s[l] = exp(s[l] - m);
      z += s[l];
    }
    for (int t = 0; t < d; ++t) {
      double acc = 0.0;
      for (int64_t l = 0; l < n; ++l) acc += (s[l] / z) * v[l * d + t];
      out[i * d + t] = acc;
    }
  }
  free(s);
}

/* ------------------------------------------------------------------------ */
/* Section 3.2.2 draws the hyperplanes of the hash at random.  When a caller */
/* gives none they come from a seed, through the counter-based generator     */
/* Philox4x64-10 of Salmon, Moraes, Dror and Shaw ("Parallel random numbers: */
/* as easy as 1, 2, 3", SC 2011): ten rounds; a round takes the 128-bit      */
/* products of words 0 and 2 with two fixed multipliers and mixes their      */
/* halves with words 1 and 3 and the key, and the key is advanced by two     */
/* Weyl increments before the next round.                                    */
/* ------------------------------------------------------------------------ */
void orc_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  const uint64_t mult0 = 0xD2E7470EE14C6C93ull, mult1 = 0xCA5A826395121157ull;
  const uint64_t weyl0 = 0x9E3779B97F4A7C15ull, weyl1 = 0xBB67AE8584CAA73Bull;
  uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    const unsigned __int128 p0 = (unsigned __int128)mult0 * x0;
    const unsigned __int128 p1 = (unsigned __int128)mult1 * x2;
    const uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    const uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    x0 = hi1 ^ x1 ^ k0;
    x1 = lo1;
    x2 = hi0 ^ x3 ^ k1;
    x3 = lo0;
    k0 += weyl0;
    k1 += weyl1;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

/* Standard normal planes[h][b][t] (flat index i over [heads][n_bits][d])   */
/* from a seed: the generator's block for counter (i / 4, 0, 0, 0) and key   */
/* (seed, 0) holds two pairs of words; pair p = (i % 4) / 2 gives           */
/* u1 = ((w_2p >> 11) + 1) 2^-53 in (0, 1] and u2 = (w_2p+1 >> 11) 2^-53 in */
/* [0, 1), and the Box-Muller transform (Box and Muller 1958) gives the two */
/* deviates r cos(phi) (even i) and r sin(phi) (odd i) with                  */
/* r = sqrt(-2 ln u1), phi = 2 pi u2, evaluated in fp64.  Planes are kept as */
/* fp32 values, so each deviate is rounded to fp32.                          */
void orc_planes(uint64_t seed, int heads, int n_bits, int d, double* planes) {
  const int64_t count = (int64_t)heads * n_bits * d;
  const double two_pi = 6.283185307179586476925286766559;
  for (int64_t i = 0; i < count; ++i) {
    const uint64_t ctr[4] = {(uint64_t)(i / 4), 0, 0, 0};
    const uint64_t key[2] = {seed, 0};
    uint64_t w[4];
    orc_philox4x64_10(ctr, key, w);
    const int p = (int)((i % 4) / 2);
    const double u1 = (double)((w[2 * p] >> 11) + 1) * 0x1.0p-53;
    const double u2 = (double)(w[2 * p + 1] >> 11) * 0x1.0p-53;
    const double r = sqrt(-2.0 * log(u1));
    const double phi = two_pi * u2;
    const double z = (i % 2 == 0) ? r * cos(phi) : r * sin(phi);
    planes[i] = (double)(float)z;
  }
}

/* ------------------------------------------------------------------------ */
/* Section 3.2.2: sign-of-random-projection hashing of the queries.           */
/* code_i bit b = [sum_t Q_it P_bt > 0] for b < n_bits.  The sum runs t = 0..d-1*/
/* in order; each product of two fp32 values is exact in fp64.               */
/* ------------------------------------------------------------------------ */
void orc_hash(const double* q, int64_t n, int d, const double* planes,
              int n_bits, uint64_t* codes) {
  for (int64_t i = 0; i < n; ++i) {
    uint64_t code = 0;
    for (int b = 0; b < n_bits; ++b) {
      double p = 0.0;
      for (int t = 0; t < d; ++t) p += q[i * d + t] * planes[b * d + t];
      if (p > 0.0) code |= (uint64_t)1 << b;
    }
    codes[i] = code;
  }
}

/* Signed projection values, used by the tests to measure how close a bit is */
/* to its decision boundary.                                                  */
void orc_projections(const double* q, int64_t n, int d, const double* planes,
                     int n_bits, double* proj) {
  for (int64_t i = 0; i < n; ++i)
    for (int b = 0; b < n_bits; ++b) {
      double p = 0.0;
      for (int t = 0; t < d; ++t) p += q[i * d + t] * planes[b * d + t];
      proj[i * n_bits + b] = p;
    }
}

/* Hamming distance between two codes. */
static int hamming(uint64_t x, uint64_t y) { return __builtin_popcountll(x ^ y); }

/* ------------------------------------------------------------------------ */
/* Section 3.2.2: K-means (Lloyd) in Hamming space on the hash codes.         */
/* L rounds of: assign each query to the centroid at the smallest Hamming     */
/* distance (tie -> smaller index), then replace each non-empty centroid by   */
/* the per-bit majority of its members (tie -> 0).  The partition S is the    */
/* assignment of the last round.  objective[2t] is sum_i ham(h_i, c_{a_i})    */
/* after the assign of round t, objective[2t+1] after its update.             */
/* ------------------------------------------------------------------------ */
void orc_kmeans(const uint64_t* h, int64_t n, int C, int L, int32_t* assign,
                uint64_t* centroids, int64_t* objective) {
  if (n <= 0) return;
  const int ce = (int64_t)C < n ? C : (int)n;
  for (int j = 0; j < ce; ++j) centroids[j] = h[((int64_t)j * n) / ce];
  int64_t* cnt = (int64_t*)calloc((size_t)ce * 64, sizeof(int64_t));
  int64_t* size = (int64_t*)calloc((size_t)ce, sizeof(int64_t));
  for (int t = 0; t < L; ++t) {
    /* assign step */
    int64_t obj = 0;
    for (int64_t i = 0; i < n; ++i) {
      int best = 0;
      int bd = hamming(h[i], centroids[0]);
      for (int j = 1; j < ce; ++j) {
        int dj = hamming(h[i], centroids[j]);
        if (dj < bd) {
          bd = dj;
          best = j;
        }
      }
      assign[i] = best;
      obj += bd;
    }
    if (objective) objective[2 * t] = obj;
    /* update step: per-bit majority of the members */
    memset(cnt, 0, sizeof(int64_t) * (size_t)ce * 64);
    memset(size, 0, sizeof(int64_t) * (size_t)ce);
    for (int64_t i = 0; i < n; ++i) {
      size[assign[i]] += 1;
      for (int b = 0; b < 64; ++b) cnt[assign[i] * 64 + b] += (int64_t)((h[i] >> b) & 1);
    }
    for (int j = 0; j < ce; ++j) {
      if (size[j] == 0) continue; /* empty cluster keeps its centroid */
      uint64_t c = 0;
      for (int b = 0; b < 64; ++b)
        if (2 * cnt[j * 64 + b] > size[j]) c |= (uint64_t)1 << b;
      centroids[j] = c;
    }
    if (objective) {
      obj = 0;
      for (int64_t i = 0; i < n; ++i) obj += hamming(h[i], centroids[assign[i]]);
      objective[2 * t + 1] = obj;
    }
  }
  free(cnt);
  free(size);
}

/* ------------------------------------------------------------------------ */
/* Section 3.2, Eq. (3): centroid of each cluster = mean of its member        */
/* queries (the real-valued queries, not their codes).  Empty clusters get a  */
/* zero row and size 0.                                                       */
/* ------------------------------------------------------------------------ */
void orc_centroids(const double* q, int64_t n, int d, const int32_t* assign,
                   int C, double* qc, int64_t* sizes) {
  for (int j = 0; j < C; ++j) {
    sizes[j] = 0;
    for (int t = 0; t < d; ++t) qc[j * d + t] = 0.0;
  }
  for (int64_t i = 0; i < n; ++i) {
    int j = assign[i];
    sizes[j] += 1;
    for (int t = 0; t < d; ++t) qc[j * d + t] += q[i * d + t];
  }
  for (int j = 0; j < C; ++j)
    if (sizes[j] > 0)
      for (int t = 0; t < d; ++t) qc[j * d + t] /= (double)sizes[j];
}

/* ------------------------------------------------------------------------ */
/* Section 3.2, Eq. (4): one row of the clustered attention matrix,           */
/* A^c_j = softmax_l(Q^c_j . K_l / sqrt(d)) over the n valid keys.            */
/* Writes the logits s_l and the probabilities a_l.                          */
/* ------------------------------------------------------------------------ */
void orc_centroid_row(const double* qcj, const double* k, int64_t n, int d,
                      double* s, double* a) {
  const double scale = 1.0 / sqrt((double)d);
  double m = -INFINITY;
  for (int64_t l = 0; l < n; ++l) {
    double dot = 0.0;
    for (int t = 0; t < d; ++t) dot += qcj[t] * k[l * d + t];
    s[l] = dot * scale;
    if (s[l] > m) m = s[l];
  }
  double z = 0.0;
  for (int64_t l = 0; l < n; ++l) {
    a[l] = exp(s[l] - m);
    z += a[l];
  }
  for (int64_t l = 0; l < n; ++l) a[l] /= z;
}

/* ------------------------------------------------------------------------ */
/* Section 3.3: the k keys of highest clustered attention for one cluster.    */
/* Keys are scanned in index order and the k best seen so far are kept        */
/* ordered by (logit descending, index ascending); a later key with an equal  */
/* logit never displaces an earlier one, so ties go to the smaller index.     */
/* The returned set is written in ascending key order.                       */
/* ------------------------------------------------------------------------ */
static int cmp_i32(const void* x, const void* y) {
  int32_t a = *(const int32_t*)x, b = *(const int32_t*)y;
  return (a > b) - (a < b);
}

int orc_topk(const double* s, int64_t n, int k, int32_t* top) {
  const int ke = (int64_t)k < n ? k : (int)n;
  if (ke <= 0) return 0;
  int cnt = 0;
  for (int64_t l = 0; l < n; ++l) {
    if (cnt == ke && !(s[l] > s[top[ke - 1]])) continue;
    int pos = cnt < ke ? cnt : ke - 1; /* slot that l will take */
    while (pos > 0 && s[l] > s[top[pos - 1]]) {
      top[pos] = top[pos - 1];
      --pos;
    }
    top[pos] = (int32_t)l;
    if (cnt < ke) ++cnt;
  }
  qsort(top, (size_t)ke, sizeof(int32_t), cmp_i32);
  return ke;
}

/* ------------------------------------------------------------------------ */
/* Section 3.2, Eq. (4)-(6): clustered attention for one (batch, head) given  */
/* the partition.  V^c_j = A^c_j V; each query takes the value of its         */
/* cluster.  vc (C x d, may be NULL) receives V^c; empty clusters give 0.     */
/* ------------------------------------------------------------------------ */
void orc_clustered_from_assign(const double* q, const double* k,
                               const double* v, int64_t n, int d,
                               const int32_t* assign, int C, double* out,
                               double* qc_out, double* vc_out) {
  double* qc = (double*)malloc(sizeof(double) * (size_t)C * d);
  int64_t* sizes = (int64_t*)malloc(sizeof(int64_t) * (size_t)C);
  double* vc = (double*)calloc((size_t)C * d, sizeof(double));
  double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  double* a = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  orc_centroids(q, n, d, assign, C, qc, sizes);
  for (int j = 0; j < C; ++j) {
    if (sizes[j] == 0) continue;
    orc_centroid_row(qc + (int64_t)j * d, k, n, d, s, a); /* Eq. (4) */
    for (int t = 0; t < d; ++t) {                          /* Eq. (5) */
      double acc = 0.0;
      for (int64_t l = 0; l < n; ++l) acc += a[l] * v[l * d + t];
      vc[j * d + t] = acc;
    }
  }
  for (int64_t i = 0; i < n; ++i) /* Eq. (6) */
    for (int t = 0; t < d; ++t) out[i * d + t] = vc[assign[i] * d + t];
  if (qc_out) memcpy(qc_out, qc, sizeof(double) * (size_t)C * d);
  if (vc_out) memcpy(vc_out, vc, sizeof(double) * (size_t)C * d);
  free(qc);
  free(sizes);
  free(vc);
  free(s);
  free(a);
}

/* ------------------------------------------------------------------------ */
/* Section 3.3 with the decomposition of the supplementary material (improved */
/* values = top-k part + rest part), for one (batch, head) given the          */
/* partition.  For query i in cluster j:                                      */
/*   m_j   = sum_{l in T_j} A^c_jl                                            */
/*   Vt_i  = m_j * sum_{l in T_j} softmax_{T_j}(Q_i . K_l / sqrt(d)) V_l      */
/*   Vb_j  = sum_{l not in T_j} A^c_jl V_l      (summed directly)             */
/*   out_i = Vt_i + Vb_j                                                      */
/* If topk_in is not NULL it supplies T (C x k, ascending, -1 padded) instead */
/* of selecting it.  topk_out / mass_out / vb_out may be NULL.                */
/* ------------------------------------------------------------------------ */
void orc_iclustered_from_assign(const double* q, const double* k,
                                const double* v, int64_t n, int d,
                                const int32_t* assign, int C, int topk,
                                const int32_t* topk_in, double* out,
                                int32_t* topk_out, double* mass_out,
                                double* vb_out) {
  const double scale = 1.0 / sqrt((double)d);
  const int ke = (int64_t)topk < n ? topk : (int)n;
  double* qc = (double*)malloc(sizeof(double) * (size_t)C * d);
  int64_t* sizes = (int64_t*)malloc(sizeof(int64_t) * (size_t)C);
  double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  double* a = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  char* in_t = (char*)malloc((size_t)(n > 0 ? n : 1));
  /* a caller-supplied set may hold up to topk entries */
  const int tcap = topk > ke ? topk : (ke > 0 ? ke : 1);
  int32_t* tj = (int32_t*)malloc(sizeof(int32_t) * (size_t)tcap);
  double* vb = (double*)malloc(sizeof(double) * (size_t)d);
  double* w = (double*)malloc(sizeof(double) * (size_t)tcap);
  orc_centroids(q, n, d, assign, C, qc, sizes);
  if (topk_out)
    for (int64_t x = 0; x < (int64_t)C * topk; ++x) topk_out[x] = -1;
  if (mass_out)
    for (int j = 0; j < C; ++j) mass_out[j] = 0.0;
  if (vb_out)
    for (int64_t x = 0; x < (int64_t)C * d; ++x) vb_out[x] = 0.0;
  for (int j = 0; j < C; ++j) {
    if (sizes[j] == 0) continue;
    orc_centroid_row(qc + (int64_t)j * d, k, n, d, s, a); /* Eq. (4) */
    int kj;
    if (topk_in) {
      kj = 0;
      while (kj < topk && topk_in[(int64_t)j * topk + kj] >= 0) {
        tj[kj] = topk_in[(int64_t)j * topk + kj];
        ++kj;
      }
    } else {
      kj = orc_topk(s, n, ke, tj); /* T_j */
    }
    memset(in_t, 0, (size_t)(n > 0 ? n : 1));
    double m = 0.0;
    for (int r = 0; r < kj; ++r) {
      in_t[tj[r]] = 1;
      m += a[tj[r]]; /* m_j */
    }
    for (int t = 0; t < d; ++t) { /* Vb_j over the keys outside T_j */
      double acc = 0.0;
      for (int64_t l = 0; l < n; ++l)
        if (!in_t[l]) acc += a[l] * v[l * d + t];
      vb[t] = acc;
    }
    for (int64_t i = 0; i < n; ++i) {
      if (assign[i] != j) continue;
      double mx = -INFINITY; /* exact logits of query i on T_j */
      for (int r = 0; r < kj; ++r) {
        double dot = 0.0;
        for (int t = 0; t < d; ++t) dot += q[i * d + t] * k[(int64_t)tj[r] * d + t];
        w[r] = dot * scale;
        if (w[r] > mx) mx = w[r];
      }
      double z = 0.0;
      for (int r = 0; r < kj; ++r) {
        w[r] = exp(w[r] - mx);
        z += w[r];
      }
      for (int t = 0; t < d; ++t) {
        double acc = 0.0;
        for (int r = 0; r < kj; ++r) acc += (w[r] / z) * v[(int64_t)tj[r] * d + t];
        out[i * d + t] = m * acc + vb[t];
      }
    }
    if (topk_out)
      for (int r = 0; r < kj; ++r) topk_out[(int64_t)j * topk + r] = tj[r];
    if (mass_out) mass_out[j] = m;
    if (vb_out)
      for (int t = 0; t < d; ++t) vb_out[(int64_t)j * d + t] = vb[t];
  }
  free(qc);
  free(sizes);
  free(s);
  free(a);
  free(in_t);
  free(tj);
  free(vb);
  free(w);
}

/* ------------------------------------------------------------------------ */
/* Dense matrices for small n (pins only).                                    */
/* Eq. (4) row of each query's cluster: ac[i][l] = A^c_{a_i, l}.              */
/* Eq. (11) improved attention:  at[i][l] = m_j softmax_{T_j}(...)_l on T_j,  */
/* A^c_jl elsewhere.                                                          */
/* ------------------------------------------------------------------------ */
void orc_dense_rows(const double* q, const double* k, int64_t n, int d,
                    const int32_t* assign, int C, int topk, double* ac,
                    double* at) {
  const double scale = 1.0 / sqrt((double)d);
  const int ke = (int64_t)topk < n ? topk : (int)n;
  double* qc = (double*)malloc(sizeof(double) * (size_t)C * d);
  int64_t* sizes = (int64_t*)malloc(sizeof(int64_t) * (size_t)C);
  double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  double* a = (double*)malloc(sizeof(double) * (size_t)C * (size_t)(n > 0 ? n : 1));
  int32_t* top = (int32_t*)malloc(sizeof(int32_t) * (size_t)C * (size_t)(ke > 0 ? ke : 1));
  int* kj = (int*)malloc(sizeof(int) * (size_t)C);
  double* w = (double*)malloc(sizeof(double) * (size_t)(ke > 0 ? ke : 1));
  orc_centroids(q, n, d, assign, C, qc, sizes);
  for (int j = 0; j < C; ++j) {
    kj[j] = 0;
    if (sizes[j] == 0) continue;
    orc_centroid_row(qc + (int64_t)j * d, k, n, d, s, a + (int64_t)j * n);
    kj[j] = orc_topk(s, n, ke, top + (int64_t)j * ke);
  }
  for (int64_t i = 0; i < n; ++i) {
    const int j = assign[i];
    const double* acj = a + (int64_t)j * n;
    for (int64_t l = 0; l < n; ++l) {
      ac[i * n + l] = acj[l];
      at[i * n + l] = acj[l];
    }
    double m = 0.0, mx = -INFINITY, z = 0.0;
    const int32_t* tj = top + (int64_t)j * ke;
    for (int r = 0; r < kj[j]; ++r) {
      m += acj[tj[r]];
      double dot = 0.0;
      for (int t = 0; t < d; ++t) dot += q[i * d + t] * k[(int64_t)tj[r] * d + t];
      w[r] = dot * scale;
      if (w[r] > mx) mx = w[r];
    }
    for (int r = 0; r < kj[j]; ++r) {
      w[r] = exp(w[r] - mx);
      z += w[r];
    }
    for (int r = 0; r < kj[j]; ++r) at[i * n + tj[r]] = m * w[r] / z;
  }
  free(qc);
  free(sizes);
  free(s);
  free(a);
  free(top);
  free(kj);
  free(w);
}

/* ------------------------------------------------------------------------ */
/* Whole forward pass over a batch: [batch][heads][N][d] row-major inputs,    */
/* lengths[batch] valid rows per sample (NULL = all N), planes [heads][n_bits]*/
/* [d].  Each (batch, head) runs independently (Section 3.2, multi-head       */
/* remark).  Rows at positions >= length are written as 0.  topk <= 0 runs    */
/* clustered attention, topk >= 1 improved clustered attention.  Every export */
/* pointer may be NULL:                                                       */
/*   codes [B][H][N] (0 on padded rows), assign [B][H][N] (-1 on padded rows),*/
/*   sizes [B][H][C], qc [B][H][C][d], topk_out [B][H][C][topk] (ascending,   */
/*   -1 padded), mass [B][H][C], vcb [B][H][C][d] (V^c for clustered, the     */
/*   rest part Vb for improved).                                              */
/* Returns 0, or -1 on invalid arguments.                                     */
/* ------------------------------------------------------------------------ */
int orc_forward(const double* q, const double* k, const double* v,
                const int32_t* lengths, int batch, int heads, int64_t N, int d,
                const double* planes, int n_bits, int C, int L, int topk,
                int num_threads, double* out, uint64_t* codes_out,
                int32_t* assign_out, int32_t* sizes_out, double* qc_out,
                int32_t* topk_out, double* mass_out, double* vcb_out) {
  if (batch < 0 || heads < 0 || N < 0 || d < 1 || n_bits < 1 || n_bits > 64 ||
      C < 1 || L < 1)
    return -1;
  const int64_t units = (int64_t)batch * heads;
  const int kk = topk > 0 ? topk : 1;
  const int nth = num_threads > 0 ? num_threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nth)
  for (int64_t u = 0; u < units; ++u) {
    const int b = (int)(u / heads), h = (int)(u % heads);
    int64_t n = lengths ? lengths[b] : N;
    if (n < 0) n = 0;
    if (n > N) n = N;
    const int64_t off = u * N * d;
    uint64_t* hc = (uint64_t*)calloc((size_t)(N > 0 ? N : 1), sizeof(uint64_t));
    int32_t* as = (int32_t*)malloc(sizeof(int32_t) * (size_t)(N > 0 ? N : 1));
    uint64_t* cent = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)C);
    double* o = out + off;
    for (int64_t x = 0; x < N * d; ++x) o[x] = 0.0;
    for (int64_t x = 0; x < N; ++x) as[x] = -1;
    double* qc = (double*)calloc((size_t)C * d, sizeof(double));
    double* vcb = (double*)calloc((size_t)C * d, sizeof(double));
    int32_t* tk = (int32_t*)malloc(sizeof(int32_t) * (size_t)C * kk);
    double* ms = (double*)calloc((size_t)C, sizeof(double));
    for (int64_t x = 0; x < (int64_t)C * kk; ++x) tk[x] = -1;
    if (n > 0) {
      orc_hash(q + off, n, d, planes + (int64_t)h * n_bits * d, n_bits, hc);
      orc_kmeans(hc, n, C, L, as, cent, NULL);
      if (topk <= 0)
        orc_clustered_from_assign(q + off, k + off, v + off, n, d, as, C, o, qc, vcb);
      else
        orc_iclustered_from_assign(q + off, k + off, v + off, n, d, as, C, topk,
                                   NULL, o, tk, ms, vcb);
    }
    if (codes_out) memcpy(codes_out + u * N, hc, sizeof(uint64_t) * (size_t)N);
    if (assign_out) memcpy(assign_out + u * N, as, sizeof(int32_t) * (size_t)N);
    if (sizes_out) {
      for (int j = 0; j < C; ++j) sizes_out[u * C + j] = 0;
      for (int64_t i = 0; i < n; ++i) sizes_out[u * C + as[i]] += 1;
    }
    if (qc_out) {
      int64_t* sz = (int64_t*)malloc(sizeof(int64_t) * (size_t)C);
      if (n > 0) orc_centroids(q + off, n, d, as, C, qc, sz);
      memcpy(qc_out + u * C * d, qc, sizeof(double) * (size_t)C * d);
      free(sz);
    }
    if (topk_out && topk > 0) memcpy(topk_out + u * C * topk, tk, sizeof(int32_t) * (size_t)C * topk);
    if (mass_out) memcpy(mass_out + u * C, ms, sizeof(double) * (size_t)C);
    if (vcb_out) memcpy(vcb_out + u * C * d, vcb, sizeof(double) * (size_t)C * d);
    free(hc);
    free(as);
    free(cent);
    free(qc);
    free(vcb);
    free(tk);
    free(ms);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Gradients.  The softmax rule: for a = softmax(s) and an upstream gradient  */
/* g_a on a, the gradient on s is a_l (g_a,l - sum_r a_r g_a,r).              */
/* ------------------------------------------------------------------------ */
static void softmax_backward(const double* a, const double* ga, int64_t n, double* gs) {
  double dot = 0.0;
  for (int64_t l = 0; l < n; ++l) dot += a[l] * ga[l];
  for (int64_t l = 0; l < n; ++l) gs[l] = a[l] * (ga[l] - dot);
}

/* Centroid part shared by both variants, for one non-empty cluster j: given */
/* the row a = A^c_j, the logit gradient gs (of s_jl = Q^c_j . K_l / sqrt(d)),*/
/* adds (1/sqrt(d)) gs_l Q^c_j to dk_l and returns dQ^c_j in dqc.            */
static void centroid_logit_backward(const double* qcj, const double* k, int64_t n, int d,
                                    const double* gs, double* dk, double* dqc) {
  const double scale = 1.0 / sqrt((double)d);
  for (int t = 0; t < d; ++t) dqc[t] = 0.0;
  for (int64_t l = 0; l < n; ++l) {
    for (int t = 0; t < d; ++t) {
      dqc[t] += scale * gs[l] * k[l * d + t];
      dk[l * d + t] += scale * gs[l] * qcj[t];
    }
  }
}

/* ------------------------------------------------------------------------ */
/* Backward pass of clustered attention (Eq. 3-6) for one (batch, head) given */
/* the partition, which is held constant.  dout, dq, dk, dv are [n][d].       */
/*   Eq. 6:  G_j = sum_{i in S_j} dout_i                                      */
/*   Eq. 5:  dV_l += sum_j A^c_jl G_j;   gA_jl = G_j . V_l                    */
/*   Eq. 4:  gs_j = softmax rule(A^c_j, gA_j); dQ^c_j, dK from s_jl           */
/*   Eq. 3:  dQ_i = dQ^c_{a_i} / |S_{a_i}|                                    */
/* ------------------------------------------------------------------------ */
void orc_clustered_backward(const double* q, const double* k, const double* v,
                            int64_t n, int d, const int32_t* assign, int C,
                            const double* dout, double* dq, double* dk, double* dv) {
  const int64_t nn = n > 0 ? n : 1;
  double* qc = (double*)malloc(sizeof(double) * (size_t)C * d);
  int64_t* sizes = (int64_t*)malloc(sizeof(int64_t) * (size_t)C);
  double* s = (double*)malloc(sizeof(double) * (size_t)nn);
  double* a = (double*)malloc(sizeof(double) * (size_t)nn);
  double* ga = (double*)malloc(sizeof(double) * (size_t)nn);
  double* gs = (double*)malloc(sizeof(double) * (size_t)nn);
  double* G = (double*)malloc(sizeof(double) * (size_t)d);
  double* dqc = (double*)calloc((size_t)C * d, sizeof(double));
  for (int64_t x = 0; x < n * d; ++x) dq[x] = dk[x] = dv[x] = 0.0;
  orc_centroids(q, n, d, assign, C, qc, sizes);
  for (int j = 0; j < C; ++j) {
    if (sizes[j] == 0) continue;
    for (int t = 0; t < d; ++t) G[t] = 0.0;
    for (int64_t i = 0; i < n; ++i)
      if (assign[i] == j)
        for (int t = 0; t < d; ++t) G[t] += dout[i * d + t];
    orc_centroid_row(qc + (int64_t)j * d, k, n, d, s, a);
    for (int64_t l = 0; l < n; ++l) {
      double g = 0.0;
      for (int t = 0; t < d; ++t) {
        dv[l * d + t] += a[l] * G[t];
        g += G[t] * v[l * d + t];
      }
      ga[l] = g;
    }
    softmax_backward(a, ga, n, gs);
    centroid_logit_backward(qc + (int64_t)j * d, k, n, d, gs, dk, dqc + (int64_t)j * d);
  }
  for (int64_t i = 0; i < n; ++i) {
    const int j = assign[i];
    for (int t = 0; t < d; ++t) dq[i * d + t] = dqc[(int64_t)j * d + t] / (double)sizes[j];
  }
  free(qc);
  free(sizes);
  free(s);
  free(a);
  free(ga);
  free(gs);
  free(G);
  free(dqc);
}

/* ------------------------------------------------------------------------ */
/* Backward pass of improved clustered attention for one (batch, head) given  */
/* the partition and the top-k sets T (C x topk, -1 padded; NULL selects them */
/* as the forward does), all held constant.  For i in S_j the forward is      */
/*   w_i   = softmax_{l in T_j}(t_il),  t_il = Q_i . K_l / sqrt(d)            */
/*   U_i   = sum_{l in T_j} w_il V_l,   out_i = m_j U_i + Vb_j,               */
/*   m_j   = sum_{l in T_j} A^c_jl,     Vb_j = sum_{l not in T_j} A^c_jl V_l, */
/* so, with g_i = dout_i:                                                     */
/*   dm_j  = sum_{i in S_j} g_i . U_i,  dVb_j = sum_{i in S_j} g_i            */
/*   top-k part:  dV_l += m_j w_il g_i;  gw_il = m_j g_i . V_l;               */
/*                gt_i = softmax rule(w_i, gw_i);  dQ_i, dK_l from t_il       */
/*   centroid part:  gA_jl = dm_j (l in T_j), dVb_j . V_l (otherwise);        */
/*                   dV_l += A^c_jl dVb_j (l not in T_j);                      */
/*                   gs_j = softmax rule(A^c_j, gA_j); dQ^c_j, dK from s_jl;  */
/*                   dQ_i += dQ^c_{a_i} / |S_{a_i}|.                          */
/* ------------------------------------------------------------------------ */
void orc_iclustered_backward(const double* q, const double* k, const double* v,
                             int64_t n, int d, const int32_t* assign, int C, int topk,
                             const int32_t* topk_in, const double* dout,
                             double* dq, double* dk, double* dv) {
  const double scale = 1.0 / sqrt((double)d);
  const int64_t nn = n > 0 ? n : 1;
  const int ke = (int64_t)topk < n ? topk : (int)n;
  const int kc = ke > 0 ? ke : 1;
  double* qc = (double*)malloc(sizeof(double) * (size_t)C * d);
  int64_t* sizes = (int64_t*)malloc(sizeof(int64_t) * (size_t)C);
  double* s = (double*)malloc(sizeof(double) * (size_t)nn);
  double* a = (double*)malloc(sizeof(double) * (size_t)nn);
  double* ga = (double*)malloc(sizeof(double) * (size_t)nn);
  double* gs = (double*)malloc(sizeof(double) * (size_t)nn);
  char* in_t = (char*)malloc((size_t)nn);
  int32_t* tj = (int32_t*)malloc(sizeof(int32_t) * (size_t)(topk > kc ? topk : kc));
  double* w = (double*)malloc(sizeof(double) * (size_t)(topk > kc ? topk : kc));
  double* gw = (double*)malloc(sizeof(double) * (size_t)(topk > kc ? topk : kc));
  double* gt = (double*)malloc(sizeof(double) * (size_t)(topk > kc ? topk : kc));
  double* U = (double*)malloc(sizeof(double) * (size_t)d);
  double* dVb = (double*)malloc(sizeof(double) * (size_t)d);
  double* dqc = (double*)calloc((size_t)C * d, sizeof(double));
  for (int64_t x = 0; x < n * d; ++x) dq[x] = dk[x] = dv[x] = 0.0;
  orc_centroids(q, n, d, assign, C, qc, sizes);
  for (int j = 0; j < C; ++j) {
    if (sizes[j] == 0) continue;
    orc_centroid_row(qc + (int64_t)j * d, k, n, d, s, a);
    int kj;
    if (topk_in) {
      kj = 0;
      while (kj < topk && topk_in[(int64_t)j * topk + kj] >= 0) {
        tj[kj] = topk_in[(int64_t)j * topk + kj];
        ++kj;
      }
    } else {
      kj = orc_topk(s, n, ke, tj);
    }
    memset(in_t, 0, (size_t)nn);
    double m = 0.0;
    for (int r = 0; r < kj; ++r) {
      in_t[tj[r]] = 1;
      m += a[tj[r]];
    }
    double dm = 0.0;
    for (int t = 0; t < d; ++t) dVb[t] = 0.0;
    /* top-k part, query by query */
    for (int64_t i = 0; i < n; ++i) {
      if (assign[i] != j) continue;
      const double* g = dout + i * d;
      double mx = -INFINITY;
      for (int r = 0; r < kj; ++r) {
        double dot = 0.0;
        for (int t = 0; t < d; ++t) dot += q[i * d + t] * k[(int64_t)tj[r] * d + t];
        w[r] = dot * scale;
        if (w[r] > mx) mx = w[r];
      }
      double z = 0.0;
      for (int r = 0; r < kj; ++r) {
        w[r] = exp(w[r] - mx);
        z += w[r];
      }
      for (int r = 0; r < kj; ++r) w[r] /= z;
      for (int t = 0; t < d; ++t) {
        double acc = 0.0;
        for (int r = 0; r < kj; ++r) acc += w[r] * v[(int64_t)tj[r] * d + t];
        U[t] = acc;
      }
      for (int t = 0; t < d; ++t) {
        dm += g[t] * U[t];
        dVb[t] += g[t];
      }
      for (int r = 0; r < kj; ++r) {
        const int64_t l = tj[r];
        double dot = 0.0;
        for (int t = 0; t < d; ++t) {
          dv[l * d + t] += m * w[r] * g[t];
          dot += g[t] * v[l * d + t];
        }
        gw[r] = m * dot;
      }
      softmax_backward(w, gw, kj, gt);
      for (int r = 0; r < kj; ++r) {
        const int64_t l = tj[r];
        for (int t = 0; t < d; ++t) {
          dq[i * d + t] += scale * gt[r] * k[l * d + t];
          dk[l * d + t] += scale * gt[r] * q[i * d + t];
        }
      }
    }
    /* centroid part */
    for (int64_t l = 0; l < n; ++l) {
      if (in_t[l]) {
        ga[l] = dm;
      } else {
        double dot = 0.0;
        for (int t = 0; t < d; ++t) {
          dv[l * d + t] += a[l] * dVb[t];
          dot += dVb[t] * v[l * d + t];
        }
        ga[l] = dot;
      }
    }
    softmax_backward(a, ga, n, gs);
    centroid_logit_backward(qc + (int64_t)j * d, k, n, d, gs, dk, dqc + (int64_t)j * d);
  }
  for (int64_t i = 0; i < n; ++i) {
    const int j = assign[i];
    for (int t = 0; t < d; ++t) dq[i * d + t] += dqc[(int64_t)j * d + t] / (double)sizes[j];
  }
  free(qc);
  free(sizes);
  free(s);
  free(a);
  free(ga);
  free(gs);
  free(in_t);
  free(tj);
  free(w);
  free(gw);
  free(gt);
  free(U);
  free(dVb);
  free(dqc);
}

/* ------------------------------------------------------------------------ */
/* Backward pass over a batch, for the partition (assign [B][H][N], -1 on     */
/* padded rows) and, for topk >= 1, the top-k sets (topk_sets [B][H][C][topk],*/
/* -1 padded) of a forward pass.  dout, dq, dk, dv are [B][H][N][d]; rows at  */
/* positions >= length get zero gradients.  Returns 0, or -1 on invalid args. */
/* ------------------------------------------------------------------------ */
int orc_backward(const double* q, const double* k, const double* v,
                 const int32_t* lengths, int batch, int heads, int64_t N, int d, int C,
                 int topk, const int32_t* assign, const int32_t* topk_sets,
                 const double* dout, int num_threads, double* dq, double* dk, double* dv) {
  if (batch < 0 || heads < 0 || N < 0 || d < 1 || C < 1) return -1;
  const int64_t units = (int64_t)batch * heads;
  const int nth = num_threads > 0 ? num_threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nth)
  for (int64_t u = 0; u < units; ++u) {
    const int b = (int)(u / heads);
    int64_t n = lengths ? lengths[b] : N;
    if (n < 0) n = 0;
    if (n > N) n = N;
    const int64_t off = u * N * d;
    for (int64_t x = 0; x < N * d; ++x) dq[off + x] = dk[off + x] = dv[off + x] = 0.0;
    if (n == 0) continue;
    if (topk <= 0)
      orc_clustered_backward(q + off, k + off, v + off, n, d, assign + u * N, C, dout + off,
                             dq + off, dk + off, dv + off);
    else
      orc_iclustered_backward(q + off, k + off, v + off, n, d, assign + u * N, C, topk,
                              topk_sets ? topk_sets + u * C * topk : NULL, dout + off,
                              dq + off, dk + off, dv + off);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Oracle-top (the comparison variant of Sec. 4.2's approximation study):     */
/* each query keeps only the k keys of highest attention, i.e. of highest     */
/* exact logit Q_i . K_l / sqrt(d) (softmax is monotone; a tie goes to the     */
/* smaller key index), and attends to those alone: out_i =                     */
/* sum_{l in T_i} softmax_{T_i}(Q_i . K_l / sqrt(d)) V_l.  The weights are     */
/* renormalised over T_i.  k_eff = min(k, n).  topk_out (n x k, may be NULL)   */
/* receives T_i in ascending key order, -1 past k_eff.                         */
/* ------------------------------------------------------------------------ */
void orc_oracle_top(const double* q, const double* k, const double* v, int64_t n,
                    int d, int topk, double* out, int32_t* topk_out) {
  const double scale = 1.0 / sqrt((double)d);
  double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  int32_t* t = (int32_t*)malloc(sizeof(int32_t) * (size_t)(topk > 0 ? topk : 1));
  for (int64_t i = 0; i < n; ++i) {
    for (int64_t l = 0; l < n; ++l) {
      double dot = 0.0;
      for (int x = 0; x < d; ++x) dot += q[i * d + x] * k[l * d + x];
      s[l] = dot * scale;
    }
    const int ke = orc_topk(s, n, topk, t); /* T_i */
    double m = -INFINITY;
    for (int r = 0; r < ke; ++r)
      if (s[t[r]] > m) m = s[t[r]];
    double z = 0.0;
    for (int r = 0; r < ke; ++r) z += exp(s[t[r]] - m);
    for (int x = 0; x < d; ++x) {
      double acc = 0.0;
      for (int r = 0; r < ke; ++r) acc += (exp(s[t[r]] - m) / z) * v[(int64_t)t[r] * d + x];
      out[i * d + x] = acc;
    }
    if (topk_out)
      for (int r = 0; r < topk; ++r) topk_out[i * topk + r] = r < ke ? t[r] : -1;
  }
  free(t);
  free(s);
}

/* Oracle-top over a padded batch [batch][heads][N][d] with per-sequence valid */
/* lengths (NULL: all N); padded rows of out are 0 and of topk_out -1.  Units  */
/* run in parallel over num_threads threads.  Returns 0, or -1 for bad sizes.  */
int orc_oracle_top_forward(const double* q, const double* k, const double* v,
                           const int32_t* lengths, int batch, int heads, int64_t N, int d,
                           int topk, int num_threads, double* out, int32_t* topk_out) {
  if (batch < 1 || heads < 1 || N < 1 || d < 1 || topk < 1) return -1;
  if (lengths)
    for (int b = 0; b < batch; ++b)
      if (lengths[b] < 0 || lengths[b] > N) return -1;
  const int64_t units = (int64_t)batch * heads;
  const int nth = num_threads > 0 ? num_threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nth)
  for (int64_t u = 0; u < units; ++u) {
    const int64_t n = lengths ? lengths[u / heads] : N;
    double* o = out + u * N * d;
    for (int64_t x = 0; x < N * d; ++x) o[x] = 0.0;
    int32_t* tk = topk_out ? topk_out + u * N * topk : NULL;
    if (tk)
      for (int64_t x = 0; x < N * topk; ++x) tk[x] = -1;
    orc_oracle_top(q + u * N * d, k + u * N * d, v + u * N * d, n, d, topk, o, tk);
  }
  return 0;
}
