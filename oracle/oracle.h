/* Declarations of the fp64 CPU oracle (test infrastructure only; see oracle.c). */
#ifndef CLUSTERED_ATTN_ORACLE_H
#define CLUSTERED_ATTN_ORACLE_H
#include <stdint.h>

void orc_full_attention(const double* q, const double* k, const double* v,
                        int64_t n, int d, double* out);
void orc_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);
void orc_planes(uint64_t seed, int heads, int n_bits, int d, double* planes);
void orc_hash(const double* q, int64_t n, int d, const double* planes,
              int n_bits, uint64_t* codes);
void orc_projections(const double* q, int64_t n, int d, const double* planes,
                     int n_bits, double* proj);
void orc_kmeans(const uint64_t* h, int64_t n, int C, int L, int32_t* assign,
                uint64_t* centroids, int64_t* objective);
void orc_centroids(const double* q, int64_t n, int d, const int32_t* assign,
                   int C, double* qc, int64_t* sizes);
void orc_centroid_row(const double* qcj, const double* k, int64_t n, int d,
                      double* s, double* a);
int orc_topk(const double* s, int64_t n, int k, int32_t* top);
void orc_clustered_from_assign(const double* q, const double* k,
                               const double* v, int64_t n, int d,
                               const int32_t* assign, int C, double* out,
                               double* qc_out, double* vc_out);
void orc_iclustered_from_assign(const double* q, const double* k,
                                const double* v, int64_t n, int d,
                                const int32_t* assign, int C, int topk,
                                const int32_t* topk_in, double* out,
                                int32_t* topk_out, double* mass_out,
                                double* vb_out);
void orc_dense_rows(const double* q, const double* k, int64_t n, int d,
                    const int32_t* assign, int C, int topk, double* ac,
                    double* at);
int orc_forward(const double* q, const double* k, const double* v,
                const int32_t* lengths, int batch, int heads, int64_t N, int d,
                const double* planes, int n_bits, int C, int L, int topk,
                int num_threads, double* out, uint64_t* codes_out,
                int32_t* assign_out, int32_t* sizes_out, double* qc_out,
                int32_t* topk_out, double* mass_out, double* vcb_out);
void orc_clustered_backward(const double* q, const double* k, const double* v,
                            int64_t n, int d, const int32_t* assign, int C,
                            const double* dout, double* dq, double* dk, double* dv);
void orc_iclustered_backward(const double* q, const double* k, const double* v,
                             int64_t n, int d, const int32_t* assign, int C, int topk,
                             const int32_t* topk_in, const double* dout,
                             double* dq, double* dk, double* dv);
int orc_backward(const double* q, const double* k, const double* v,
                 const int32_t* lengths, int batch, int heads, int64_t N, int d, int C,
                 int topk, const int32_t* assign, const int32_t* topk_sets,
                 const double* dout, int num_threads, double* dq, double* dk, double* dv);
void orc_oracle_top(const double* q, const double* k, const double* v, int64_t n,
                    int d, int topk, double* out, int32_t* topk_out);
int orc_oracle_top_forward(const double* q, const double* k, const double* v,
                           const int32_t* lengths, int batch, int heads, int64_t N, int d,
                           int topk, int num_threads, double* out, int32_t* topk_out);
#endif
