/*
 * clustered_attn.h -- C ABI of the gfx950 (MI355X) library for the forward
 * pass of clustered and improved-clustered attention
 * (Vyas, Katharopoulos, Fleuret, "Fast Transformers with Clustered Attention").
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * - q, k, v and out are DEVICE pointers to contiguous row-major tensors of
 *   shape [batch][heads][n][d] with element type `dtype` (CA_F32 or CA_BF16,
 *   the same for all four).  A (batch, head) pair is a "unit"; units are
 *   independent (Section 3.2: each head clusters its own queries).
 * - lengths is NULL (every row valid) or a DEVICE pointer to int32[batch]:
 *   only rows 0..lengths[b]-1 of sample b are queries/keys.  Values are
 *   clamped to [0, n] on the device.  Keys past the length get no attention,
 *   queries past it are not hashed or clustered, and their output rows are
 *   written as 0.
 * - planes is NULL or a DEVICE pointer to fp32[heads][n_bits][d]: the random
 *   hyperplanes of the sign-random-projection hash (Section 3.2.2).  Any fp32
 *   values work; the projections are evaluated in fp64, where each product
 *   is exact.  When planes is NULL the library draws them from `seed` into
 *   the workspace: entry i of the flat [heads][n_bits][d] order is a
 *   standard normal deviate from block i / 4 of the counter-based generator
 *   Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011; counter
 *   (i / 4, 0, 0, 0), key (seed, 0)), whose words (2p, 2p + 1),
 *   p = (i mod 4) / 2, give u1 = ((w >> 11) + 1) 2^-53 and u2 = (w >> 11)
 *   2^-53 and, by the Box-Muller transform in fp64, the deviates
 *   sqrt(-2 ln u1) cos(2 pi u2) (even i) and sqrt(-2 ln u1) sin(2 pi u2)
 *   (odd i), rounded to fp32.  The same seed gives the same planes for
 *   every call and sequence length; `seed` is ignored when planes is given.
 * - C = n_clusters, B = n_bits, L = lloyd_iters, k = topk are the method's
 *   hyper-parameters (Sections 3.2.2 and 3.3).  Per unit the library uses
 *   C_eff = min(C, length) clusters and k_eff = min(k, length) keys.
 * - workspace is a DEVICE buffer of at least ca_workspace_bytes(...) bytes,
 *   owned by the caller and 256-byte aligned; its contents on entry do not
 *   matter.  On exit it holds the forward pass's state (partition,
 *   centroids, top-k sets, softmax statistics), which the backward entry
 *   points below read; nothing else about its contents is specified.  The
 *   library allocates no device memory in a forward or backward call.
 * - stream is a hipStream_t (NULL = the null stream).  All work is enqueued
 *   on it and the call returns without synchronising.  Arguments are
 *   validated on the host before anything is enqueued: on an error nothing
 *   is launched.  A fault inside a kernel surfaces at the caller's next
 *   synchronisation.
 * - Results are deterministic: identical inputs give bitwise identical
 *   outputs (no floating-point atomics are used).
 * - Return value: CA_OK, or a negative CA_ERR_* code; ca_last_error() then
 *   returns a message for the calling thread.  No C++ exception crosses this
 *   interface.
 *
 * Supported sizes: d in {32, 64}; 1 <= n_bits <= 64; 1 <= C <= 256;
 * 1 <= L <= 1000; 1 <= k <= 128; 1 <= n <= 1048576; 1 <= batch*heads <= 65535
 * and batch*heads*n < 2^31.
 *
 * The backward entry points (clustered_attention_bwd, iclustered_attention_bwd)
 * follow the same conventions; their gradient outputs are fp32 for both
 * input dtypes.
 */
#ifndef CLUSTERED_ATTN_H
#define CLUSTERED_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CA_OK 0
#define CA_ERR_INVALID_ARG (-1) /* null required pointer, non-positive size, bad enum */
#define CA_ERR_UNSUPPORTED (-2) /* size outside the supported ranges above          */
#define CA_ERR_WORKSPACE (-3)   /* workspace NULL or smaller than required          */
#define CA_ERR_HIP (-4)         /* a HIP runtime call failed                        */

#define CA_F32 0
#define CA_BF16 1

/*
 * Optional stage inputs and outputs (all DEVICE pointers, each may be NULL).
 * An "_in" pointer replaces the stage that would compute it, which is how the
 * stages are tested one at a time; an "_out" pointer receives a copy of an
 * intermediate result.  Shapes use U = batch*heads and the unit order of q.
 *
 *   codes_in    uint64[U][n]  hash codes; skips hashing.  Bits at positions
 *                             >= n_bits are ignored.
 *   assign_in   int32[U][n]   cluster of each valid query, in
 *                             [0, C_eff); skips hashing and K-means.
 *   topk_in     int32[U][C][k] top-k key set of each cluster, ascending and
 *                             -1 padded, each entry < length; skips the
 *                             top-k selection (improved variant only).
 *   codes_out   uint64[U][n]  hash codes (Section 3.2.2); 0 on padded rows.
 *   assign_out  int32[U][n]   final cluster of each query (the assignment of
 *                             the L-th Lloyd round); -1 on padded rows.
 *   sizes_out   int32[U][C]   members per cluster.
 *   centroids_out float[U][C][d] query centroids Q^c (Eq. 3); 0 when empty.
 *   topk_out    int32[U][C][k] top-k set T_j (Section 3.3), ascending, -1
 *                             padded and all -1 for empty clusters.
 *   mass_out    float[U][C]   clustered attention mass on T_j (Section 3.3).
 *   values_out  float[U][C][d] V^c = A^c V (Eq. 5) for the clustered variant;
 *                             for the improved variant the part of A^c V
 *                             over the keys outside T_j (supplementary
 *                             decomposition of the improved values).
 *   planes_out  float[heads][n_bits][d] the hash planes used: the caller's,
 *                             or those drawn from the seed.
 */
typedef struct ca_aux {
  const uint64_t* codes_in;
  const int32_t* assign_in;
  const int32_t* topk_in;
  uint64_t* codes_out;
  int32_t* assign_out;
  int32_t* sizes_out;
  float* centroids_out;
  int32_t* topk_out;
  float* mass_out;
  float* values_out;
  float* planes_out;
} ca_aux;

/*
 * Bytes of workspace that clustered_attention_fwd (topk = 0) or
 * iclustered_attention_fwd (topk >= 1) needs for these sizes (n_bits sizes
 * the room for planes drawn from a seed).  Returns 0 if the sizes are
 * invalid or unsupported.
 */
size_t ca_workspace_bytes(int batch, int heads, int n, int d, int dtype,
                          int n_clusters, int n_bits, int topk);

/*
 * Clustered attention (Section 3.2, Eqs. 3-6), one call for all units:
 *   1. hash each valid query to an n_bits code by the signs of its
 *      projections on the planes (Section 3.2.2);
 *   2. run L rounds of K-means in Hamming space on the codes (assign to the
 *      nearest binary centroid, ties to the smaller index; replace each
 *      non-empty centroid by the per-bit majority of its members, ties to 0;
 *      initial centroids: the codes of queries floor(j*length/C_eff));
 *   3. Q^c_j = mean of the member queries (Eq. 3);
 *   4. A^c = softmax(Q^c K^T / sqrt(d)) over the valid keys (Eq. 4),
 *      V^c = A^c V (Eq. 5);
 *   5. out_i = V^c of the cluster of query i (Eq. 6).
 */
int clustered_attention_fwd(const void* q, const void* k, const void* v,
                            const int32_t* lengths, const float* planes,
                            int batch, int heads, int n, int d, int dtype,
                            int n_clusters, int n_bits, int lloyd_iters,
                            uint64_t seed, void* out, void* workspace,
                            size_t workspace_bytes, const ca_aux* aux,
                            void* stream);

/*
 * Improved clustered attention (Section 3.3, Eq. 11), steps 1-4 as above and
 * then, per cluster j:
 *   5. T_j = the k_eff keys with the largest centroid logit (ties to the
 *      smaller key index), m_j = sum of A^c_jl over l in T_j;
 *   6. for each member query i:
 *        out_i = m_j * sum_{l in T_j} softmax_{T_j}(Q_i K_l / sqrt(d)) V_l
 *              + sum_{l not in T_j} A^c_jl V_l
 *      (the decomposition of A^t V given in the supplementary material).
 */
int iclustered_attention_fwd(const void* q, const void* k, const void* v,
                             const int32_t* lengths, const float* planes,
                             int batch, int heads, int n, int d, int dtype,
                             int n_clusters, int n_bits, int lloyd_iters,
                             uint64_t seed, int topk, void* out,
                             void* workspace, size_t workspace_bytes,
                             const ca_aux* aux, void* stream);

/*
 * Backward pass.  The paper trains through the operator (Section 4) without
 * writing its gradient; here the partition (Section 3.2.2) and the top-k
 * sets (Section 3.3) are discrete and held constant, and the gradient flows
 * through the centroids (Eq. 3), the centroid softmax and values (Eqs. 4-5),
 * the broadcast (Eq. 6) and, for the improved variant, through the exact
 * top-k logits, the mass m_j and the rest part of the supplementary
 * decomposition (all three depend on Q, K and V).
 *
 * Bytes of bwd_workspace that clustered_attention_bwd (topk = 0) or
 * iclustered_attention_bwd (topk >= 1) needs; 0 for invalid sizes.
 */
size_t ca_backward_workspace_bytes(int batch, int heads, int n, int d, int dtype,
                                   int n_clusters, int topk);

/*
 * Gradients of the clustered attention forward pass (the same arguments as
 * clustered_attention_fwd) with respect to q, k and v, for the output
 * gradient dout ([batch][heads][n][d], element type dtype, DEVICE):
 *   G_j = sum of dout_i over the members of cluster j;
 *   dV_l = sum_j A^c_jl G_j;  dS_jl = A^c_jl (G_j . V_l - G_j . V^c_j);
 *   dK_l = sum_j dS_jl Q^c_j / sqrt(d);  dQ_i = sum_l dS_{a_i,l} K_l / (sqrt(d) |S_{a_i}|).
 * workspace must be the buffer of the forward call made last with the same
 * q, k, v, lengths and sizes (clustered_attention_fwd, n_clusters as given),
 * unchanged since; it is only read.  dq, dk, dv are DEVICE fp32
 * [batch][heads][n][d], written fully (rows past a length get 0).
 * bwd_workspace is a caller-owned DEVICE buffer of at least
 * ca_backward_workspace_bytes bytes, 256-byte aligned, contents irrelevant.
 * Enqueued on stream; validation before any launch; deterministic (no
 * floating-point atomics).
 */
int clustered_attention_bwd(const void* q, const void* k, const void* v,
                            const int32_t* lengths, int batch, int heads, int n,
                            int d, int dtype, int n_clusters, const void* dout,
                            float* dq, float* dk, float* dv, const void* workspace,
                            size_t workspace_bytes, void* bwd_workspace,
                            size_t bwd_workspace_bytes, void* stream);

/*
 * Gradients of the improved clustered attention forward pass (Section 3.3,
 * Eq. 11 in its supplementary decomposition), with the top-k sets of the
 * forward call held constant.  For query i in cluster j, with
 * w_i = softmax_{T_j}(Q_i K_l / sqrt(d)), U_i = sum_{l in T_j} w_il V_l and
 * g_i = dout_i:
 *   dm_j = sum_i g_i . U_i;  gt_il = m_j w_il (g_i . V_l - g_i . U_i);
 *   top-k part:    dQ_i += sum_l gt_il K_l / sqrt(d),
 *                  dK_l += sum_i gt_il Q_i / sqrt(d),  dV_l += m_j sum_i w_il g_i;
 *   centroid part: gA_jl = dm_j on T_j, G_j . V_l elsewhere;
 *                  dV_l += sum_j [l not in T_j] A^c_jl G_j;
 *                  dS_jl = A^c_jl (gA_jl - sum_l' A^c_jl' gA_jl'), then dQ^c,
 *                  dK and dQ as for the clustered variant.
 * workspace must be that of the last iclustered_attention_fwd call with the
 * same inputs, n_clusters and topk; other arguments as for
 * clustered_attention_bwd.  The top-k parts of dK_l and dV_l are summed over
 * the sets that hold key l as 64-bit fixed-point integers (units of 2^-32),
 * which makes the result independent of their order; a term above 2^22 in
 * magnitude, or one that is not finite, cannot be held, and the dK or dV
 * entry it belongs to is then written as NaN.
 */
int iclustered_attention_bwd(const void* q, const void* k, const void* v,
                             const int32_t* lengths, int batch, int heads, int n,
                             int d, int dtype, int n_clusters, int topk,
                             const void* dout, float* dq, float* dk, float* dv,
                             const void* workspace, size_t workspace_bytes,
                             void* bwd_workspace, size_t bwd_workspace_bytes,
                             void* stream);

/*
 * Oracle-top attention: the comparison variant of the approximation study
 * (Section 4.2) in which each query keeps only its k keys of highest
 * attention.  For every valid query i of a unit, T_i is the set of
 * k_eff = min(k, length) keys with the largest logits Q_i . K_l / sqrt(d)
 * (a tie goes to the smaller key index), and
 *   out_i = sum_{l in T_i} softmax_{T_i}(Q_i . K_l / sqrt(d))_l V_l,
 * the softmax renormalised over T_i.  No hashing or clustering takes place;
 * the cost is that of exact attention, O(n^2 d) per unit.
 * q, k, v, out, lengths, dtype, stream: as above.  topk_out is NULL or a
 * DEVICE int32[batch][heads][n][topk]: T_i in ascending key order, -1 past
 * k_eff and for padded rows.  workspace: at least
 * ca_oracle_top_workspace_bytes(...) bytes, 256-byte aligned, contents
 * irrelevant; it grows as n * ceil(n / 1024) * topk per unit.
 * Sizes as above (n_clusters, n_bits and lloyd_iters do not apply).
 * Passing the same pointer as q and k gives the shared-QK input mode of the
 * same study (keys equal to the queries); every entry point of this library
 * accepts that aliasing, since q and k are only read.
 */
size_t ca_oracle_top_workspace_bytes(int batch, int heads, int n, int d, int dtype,
                                     int topk);
int oracle_top_attention_fwd(const void* q, const void* k, const void* v,
                             const int32_t* lengths, int batch, int heads, int n,
                             int d, int dtype, int topk, void* out, int32_t* topk_out,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * improved clustered attention forward of iclustered_attention_fwd, with the
 * same arguments and results but no workspace argument.  Its scratch is a
 * device array of CA_NOALLOC_SCRATCH_BYTES bytes inside the library, one per
 * GPU, held until the process ends; the call allocates nothing (no hipMalloc,
 * no hipFree, no allocating library routine).  Sizes whose workspace
 * (ca_workspace_bytes with the same arguments) exceeds that maximum are
 * rejected with CA_ERR_UNSUPPORTED before anything is enqueued.  Every call
 * on one GPU uses that GPU's single array, which keeps the last call's
 * contents (nothing in it needs to start at zero): calls that overlap on one
 * GPU, on different streams or threads, race and give wrong results; calls
 * on one stream are ordered and safe.  As with the workspace of the other
 * entry point, the array then holds the call's forward state, but no
 * backward entry point can be pointed at it.
 */
#define CA_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)
int iclustered_attention_fwd_noalloc(const void* q, const void* k, const void* v,
                                     const int32_t* lengths, const float* planes,
                                     int batch, int heads, int n, int d, int dtype,
                                     int n_clusters, int n_bits, int lloyd_iters,
                                     uint64_t seed, int topk, void* out,
                                     const ca_aux* aux, void* stream);

/* Message describing the last non-zero status returned on this thread. */
const char* ca_last_error(void);

/* Library version, major*10000 + minor*100 + patch. */
int ca_version(void);

/*
 * Stages of a forward call, for ca_time_next_stage.
 *   CA_KERNEL_HASH           hashing of the queries (Section 3.2.2)
 *   CA_KERNEL_KMEANS         the L Lloyd rounds of Hamming K-means
 *   CA_KERNEL_CENTROIDS      query centroids (Eq. 3)
 *   CA_KERNEL_CENTROID_ATTN  centroid attention, top-k and mass (Eqs. 4-5, Section 3.3);
 *                            in an oracle-top call, its whole work
 *   CA_KERNEL_OUTPUT         broadcast (Eq. 6) or the improved per-query part
 *   CA_KERNEL_BWD_CENTROID   (backward calls) the centroid part of the
 *                            gradient: dK, dV and the dQ^c partials
 *   CA_KERNEL_ATTN_TILE      the centroid-attention kernel alone (Eqs. 4-5 on
 *                            the matrix cores), without the merge of several
 *                            key chunks that CA_KERNEL_CENTROID_ATTN includes
 */
#define CA_KERNEL_HASH 1
#define CA_KERNEL_KMEANS 2
#define CA_KERNEL_CENTROIDS 3
#define CA_KERNEL_CENTROID_ATTN 4
#define CA_KERNEL_OUTPUT 5
#define CA_KERNEL_BWD_CENTROID 6
#define CA_KERNEL_ATTN_TILE 7

/*
 * Profiling hook for callers that time one stage with HIP events: in the
 * next forward call (backward call for CA_KERNEL_BWD_CENTROID) made by this
 * thread, hipEventRecord(start_event) is
 * enqueued on the call's stream just before the stage's kernels and
 * hipEventRecord(stop_event) just after them; the hook is then disarmed.
 * start_event and stop_event are hipEvent_t owned by the caller.  stage 0
 * disarms it.  Returns CA_OK or CA_ERR_INVALID_ARG.
 */
int ca_time_next_stage(int stage, void* start_event, void* stop_event);

/*
 * Chooses the K-means driver for later calls in this process: 0 automatic
 * (default), 1 one workgroup per unit (used only when n <= 4096), 2 one
 * kernel pair per Lloyd round, 3 one cooperative launch for all rounds (used
 * only when all its workgroups fit on the device at once, otherwise 2), whose
 * workgroups also form the per-workgroup centroid sums when its grid covers
 * every compute unit; 4 and 5 are 3 with those sums always formed by the
 * K-means kernel (4) or always by a separate kernel (5).  All give identical
 * partitions and centroids within fp32 rounding; the switch exists so that
 * tests cover every driver and benchmarks can compare them.  Returns CA_OK or
 * CA_ERR_INVALID_ARG.
 */
int ca_set_kmeans_path(int path);

#ifdef __cplusplus
}
#endif

#endif /* CLUSTERED_ATTN_H */
