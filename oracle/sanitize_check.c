/*
 * Driver that runs every entry point of the fp64 oracle once on small ragged
 * inputs, for a build with AddressSanitizer and UndefinedBehaviorSanitizer
 * (TEST INFRASTRUCTURE ONLY; the CPU test-suite compiles and runs it).
 *
 * It covers the paths with the most hand-made indexing: padded and empty
 * sequences (lengths 0, 1, a ragged one and the full length), C larger than
 * a sequence, k larger than a sequence, a caller-supplied top-k set that is
 * shorter than k (-1 terminated), n_bits = 64, and both backward variants
 * fed with the forward pass's own partition and top-k sets, and the seeded
 * plane generator.  The values are
 * irrelevant here: the sanitizers check the memory accesses and the integer
 * arithmetic.  Exit status 0 and the line "sanitize ok" mean that no check
 * fired (the build aborts on the first report).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static uint64_t g_state = 0x2007048250000001ull;

/* splitmix64 (Steele, Lea, Flood 2014): a uniform 64-bit stream */
static uint64_t next_u64(void) {
  uint64_t z = (g_state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

/* uniform in [-2, 2) */
static double next_val(void) { return (double)(next_u64() >> 11) * 0x1.0p-53 * 4.0 - 2.0; }

static double* make(size_t count) {
  double* x = (double*)malloc(sizeof(double) * (count ? count : 1));
  for (size_t i = 0; i < count; ++i) x[i] = next_val();
  return x;
}

static int run_case(int batch, int heads, int64_t N, int d, int C, int n_bits, int L, int topk,
                    const int32_t* lengths, int threads) {
  const size_t rows = (size_t)batch * heads * (size_t)N;
  const size_t U = (size_t)batch * heads;
  const int kk = topk > 0 ? topk : 1;
  double* q = make(rows * d);
  double* k = make(rows * d);
  double* v = make(rows * d);
  double* dout = make(rows * d);
  double* planes = make((size_t)heads * n_bits * d);
  double* out = (double*)malloc(sizeof(double) * rows * d);
  uint64_t* codes = (uint64_t*)malloc(sizeof(uint64_t) * rows);
  int32_t* assign = (int32_t*)malloc(sizeof(int32_t) * rows);
  int32_t* sizes = (int32_t*)malloc(sizeof(int32_t) * U * C);
  double* qc = (double*)malloc(sizeof(double) * U * C * d);
  int32_t* tk = (int32_t*)malloc(sizeof(int32_t) * U * C * kk);
  double* mass = (double*)malloc(sizeof(double) * U * C);
  double* vcb = (double*)malloc(sizeof(double) * U * C * d);
  double* dq = (double*)malloc(sizeof(double) * rows * d);
  double* dk = (double*)malloc(sizeof(double) * rows * d);
  double* dv = (double*)malloc(sizeof(double) * rows * d);
  int32_t* otop = (int32_t*)malloc(sizeof(int32_t) * rows * kk);
  int rc = 0;
  for (int variant = 0; variant < 2 && rc == 0; ++variant) {
    const int t = variant ? topk : 0;
    rc |= orc_forward(q, k, v, lengths, batch, heads, N, d, planes, n_bits, C, L, t, threads, out,
                      codes, assign, sizes, qc, t > 0 ? tk : NULL, mass, vcb);
    rc |= orc_backward(q, k, v, lengths, batch, heads, N, d, C, t, assign, t > 0 ? tk : NULL, dout,
                       threads, dq, dk, dv);
    /* the backward pass selecting its own top-k sets */
    if (t > 0)
      rc |= orc_backward(q, k, v, lengths, batch, heads, N, d, C, t, assign, NULL, dout, threads,
                         dq, dk, dv);
  }
  if (topk > 0 && rc == 0) rc |= orc_oracle_top_forward(q, k, v, lengths, batch, heads, N, d, topk,
                                                        threads, out, otop);
  free(q); free(k); free(v); free(dout); free(planes); free(out); free(codes); free(assign);
  free(sizes); free(qc); free(tk); free(mass); free(vcb); free(dq); free(dk); free(dv); free(otop);
  return rc;
}

/* The per-unit functions on one sequence of n rows, including a top-k set   */
/* shorter than k and the dense matrices.                                    */
static int run_unit(int64_t n, int d, int C, int n_bits, int L, int topk) {
  const int kk = topk > 0 ? topk : 1;
  double* q = make((size_t)n * d);
  double* k = make((size_t)n * d);
  double* v = make((size_t)n * d);
  double* dout = make((size_t)n * d);
  double* planes = make((size_t)n_bits * d);
  double* out = (double*)malloc(sizeof(double) * (size_t)n * d);
  double* proj = (double*)malloc(sizeof(double) * (size_t)n * n_bits);
  uint64_t* codes = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)n);
  int32_t* assign = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
  uint64_t* cent = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)C);
  int64_t* obj = (int64_t*)malloc(sizeof(int64_t) * 2 * (size_t)L);
  double* qc = (double*)malloc(sizeof(double) * (size_t)C * d);
  int64_t* sizes = (int64_t*)malloc(sizeof(int64_t) * (size_t)C);
  double* s = (double*)malloc(sizeof(double) * (size_t)n);
  double* a = (double*)malloc(sizeof(double) * (size_t)n);
  int32_t* top = (int32_t*)malloc(sizeof(int32_t) * (size_t)kk);
  int32_t* tin = (int32_t*)malloc(sizeof(int32_t) * (size_t)C * kk);
  int32_t* tout = (int32_t*)malloc(sizeof(int32_t) * (size_t)C * kk);
  double* mass = (double*)malloc(sizeof(double) * (size_t)C);
  double* vb = (double*)malloc(sizeof(double) * (size_t)C * d);
  double* dq = (double*)malloc(sizeof(double) * (size_t)n * d);
  double* dk = (double*)malloc(sizeof(double) * (size_t)n * d);
  double* dv = (double*)malloc(sizeof(double) * (size_t)n * d);
  double* ac = (double*)malloc(sizeof(double) * (size_t)n * n);
  double* at = (double*)malloc(sizeof(double) * (size_t)n * n);
  orc_full_attention(q, k, v, n, d, out);
  orc_projections(q, n, d, planes, n_bits, proj);
  orc_hash(q, n, d, planes, n_bits, codes);
  orc_kmeans(codes, n, C, L, assign, cent, obj);
  const int ce = (int64_t)C < n ? C : (int)n;
  orc_centroids(q, n, d, assign, ce, qc, sizes);
  orc_centroid_row(qc, k, n, d, s, a);
  (void)orc_topk(s, n, topk, top);
  orc_clustered_from_assign(q, k, v, n, d, assign, ce, out, qc, vb);
  orc_iclustered_from_assign(q, k, v, n, d, assign, ce, topk, NULL, out, tout, mass, vb);
  /* caller-supplied sets: the first half of each selected set, -1 terminated */
  for (int x = 0; x < C * kk; ++x) tin[x] = -1;
  for (int j = 0; j < ce; ++j)
    for (int r = 0; r < kk / 2; ++r) tin[j * kk + r] = tout[j * kk + r];
  orc_iclustered_from_assign(q, k, v, n, d, assign, ce, topk, tin, out, tout, mass, vb);
  orc_clustered_backward(q, k, v, n, d, assign, ce, dout, dq, dk, dv);
  orc_iclustered_backward(q, k, v, n, d, assign, ce, topk, tin, dout, dq, dk, dv);
  orc_iclustered_backward(q, k, v, n, d, assign, ce, topk, NULL, dout, dq, dk, dv);
  orc_dense_rows(q, k, n, d, assign, ce, topk, ac, at);
  orc_oracle_top(q, k, v, n, d, topk, out, NULL);
  free(q); free(k); free(v); free(dout); free(planes); free(out); free(proj); free(codes);
  free(assign); free(cent); free(obj); free(qc); free(sizes); free(s); free(a); free(top);
  free(tin); free(tout); free(mass); free(vb); free(dq); free(dk); free(dv); free(ac); free(at);
  return 0;
}

/* The seeded planes, including a count that is not a multiple of a block. */
static int run_planes(void) {
  double* p = (double*)malloc(sizeof(double) * 3 * 7 * 5);
  orc_planes(0xffffffffffffffffull, 3, 7, 5, p);
  const uint64_t ctr[4] = {~0ull, ~0ull, ~0ull, ~0ull}, key[2] = {~0ull, 1};
  uint64_t w[4];
  orc_philox4x64_10(ctr, key, w);
  int ok = 1;
  for (int i = 0; i < 3 * 7 * 5; ++i) ok &= isfinite(p[i]) ? 1 : 0;
  free(p);
  return ok ? 0 : 1;
}

int main(void) {
  const int32_t lengths[4] = {37, 0, 1, 64};
  int rc = run_planes();
  rc |= run_case(4, 2, 64, 8, 9, 63, 4, 5, lengths, 2);    /* ragged, C and k above some lengths */
  rc |= run_case(4, 1, 64, 4, 80, 64, 2, 100, lengths, 1); /* C > N, k > N, n_bits = 64 */
  rc |= run_case(1, 3, 17, 16, 1, 1, 1, 1, NULL, 3);       /* C = 1, B = 1, L = 1, k = 1 */
  rc |= run_unit(50, 8, 6, 63, 3, 7);
  rc |= run_unit(5, 4, 9, 64, 2, 12);                      /* C and k above n */
  rc |= run_unit(1, 32, 1, 1, 1, 1);
  if (rc != 0) {
    fprintf(stderr, "an oracle entry point rejected its arguments\n");
    return 1;
  }
  printf("sanitize ok\n");
  return 0;
}
