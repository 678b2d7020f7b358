// Host-side launchers of the gfx950 kernels (internal to the library).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ca {

// Problem description shared by the launchers.
struct Problem {
  int batch, heads, n, d, dtype;   // n = padded length N
  int C, n_bits, L, topk;          // topk = 0 for the clustered variant
  const void* q;
  const void* k;
  const void* v;
  const int32_t* lengths;          // device, may be null
  const float* planes;             // device [heads][n_bits][d]
  void* out;
  int units() const { return batch * heads; }
};

// Keys per chunk of the centroid-attention kernel.
constexpr int kChunk = 1024;
// Largest n handled by the one-workgroup-per-unit K-means.
constexpr int kKmLdsMaxN = 4096;
// Queries per workgroup of the multi-workgroup K-means.
constexpr int kKmBlockQ = 1024;
// Queries per workgroup of the CSR build.
constexpr int kCsrBlockQ = 256;
// Queries per workgroup of the cooperative K-means (codes resident in LDS):
// 1024 or 2048, the smaller one whose grid the device holds at once.
constexpr int kCoopMinQ = 1024;
constexpr int kCoopMaxQ = 2048;
// Workgroups of the cooperative K-means that the workspace is sized for.
constexpr int kCoopMaxWgs = 512;
inline int coop_max_blocks(int n, int units) {
  const int by_len = (n + kCoopMinQ - 1) / kCoopMinQ;
  const int by_grid = units > 0 ? (kCoopMaxWgs / units > 0 ? kCoopMaxWgs / units : 1) : 1;
  return by_len < by_grid ? by_len : by_grid;
}
// Ints per unit of the cooperative K-means' two arrival words (64-bit each,
// 8-byte aligned); the kernel that runs before it (hashing, or the copy of
// given codes) sets them and both count tables to zero.
constexpr int kSyncInts = 4;
// Words per unit of a count table of the cooperative K-means.
int coop_table_stride(int C);

// Device buffers carved from the caller's workspace.
struct Workspace {
  uint64_t* codes;      // [U][N]
  int32_t* assign;      // [U][N]
  int32_t* members;     // [U][N]   CSR member lists, ascending query index per cluster
  int32_t* offsets;     // [U][C+1]
  int32_t* sizes;       // [U][C]
  uint64_t* cent;       // [2][U][C] centroid codes (multi-workgroup K-means)
  uint32_t* part;       // [U][nblk][C][32] packed 16-bit bit-pair counts
  int32_t* part_sizes;  // [U][nblk][C]
  int32_t* csr_cnt;     // [U][ncsr][C] per-block counts, then per-block bases
  float* qc;            // [U][C][d]
  float* pm;            // [U][C][nchunk]
  float* pz;            // [U][C][nchunk]
  float* pacc;          // [U][C][nchunk][d]
  int32_t* cand_idx;    // [U][C][nchunk][k]
  float* cand_val;      // [U][C][nchunk][k]
  int32_t* topk;        // [U][C][k]
  float* mass;          // [U][C]
  float* vcb;           // [U][C][d]
  float* stats;         // [U][C][2] row maximum and normaliser of the centroid softmax
  int32_t* sync;        // [U][kSyncInts] arrival counters of the cooperative K-means
  uint64_t* ctab;       // [U][2][C * 33] running count tables of the cooperative K-means
  int32_t* cbases;      // [U][ncoop][C] first member position of each (block, cluster)
  int32_t* clsizes;     // [U][ncoop][C] members of each (block, cluster)
  double* qc_part;      // [U][C][ncoop][d] per-block centroid sums (used: n / coop_q blocks)
  float* planes;        // [heads][n_bits][d] hash planes drawn from the seed (caller gave none)
  int nblk;             // ceil(N / kKmBlockQ)
  int ncsr;             // ceil(N / kCsrBlockQ)
  int nchunk;           // ceil(N / kChunk)
  int ncoop;            // cooperative K-means blocks the workspace holds per unit
  int coop_q;           // queries per cooperative block of this call (0: not used)
  int coop_sums;        // 1: the cooperative K-means forms the blocks' centroid sums itself
};

// Carves the workspace; returns the bytes needed (ws may be null to only size it).
size_t carve_workspace(const Problem& p, void* base, Workspace* ws);
// Oracle-top (p.C = p.n, one row per query): carves topk [U][N][k] and, for
// several key chunks, cand_idx and cand_val [U][N][nchunk][k]; the other
// fields are null.
size_t carve_otop_workspace(const Problem& p, void* base, Workspace* ws);
// Oracle-top outputs and top-k sets (into ws.topk).
hipError_t launch_oracle_top(const Problem& p, const Workspace& ws, hipStream_t s);

// Hash planes [heads][n_bits][d] drawn from seed (when the caller gives none).
hipError_t launch_planes(const Problem& p, uint64_t seed, float* planes, hipStream_t s);
// Hashing; also writes 0 to the output rows past each sequence's length and
// zeroes ws.sync.
hipError_t launch_hash(const Problem& p, const Workspace& ws, hipStream_t s);
hipError_t launch_load_codes(const Problem& p, const uint64_t* codes_in, const Workspace& ws,
                             hipStream_t s);
// One workgroup per unit (n <= kKmLdsMaxN): hashing (or the given codes),
// K-means, member lists (sizes, offsets, members) and centroids; also zeroes
// the output rows past each sequence's length.
hipError_t launch_cluster_lds(const Problem& p, const uint64_t* codes_in, const Workspace& ws,
                              hipStream_t s);
// Multi-workgroup K-means on ws.codes, one launch pair per round: writes the
// assignments of valid rows.
hipError_t launch_kmeans(const Problem& p, const Workspace& ws, hipStream_t s);
// Cooperative K-means on ws.codes (ws.sync zero), all rounds in one launch:
// assignments (-1 on padded rows), sizes, offsets, member lists and either
// each block's fp64 centroid sums (ws.coop_sums) or the per-block member
// ranges from which launch_coop_centroids forms them.
hipError_t launch_kmeans_coop(const Problem& p, const Workspace& ws, hipStream_t s);
// Centroids (Eq. 3) after launch_kmeans_coop: per-block fp64 partial sums
// (unless the K-means formed them), then added in block order.
hipError_t launch_coop_centroids(const Problem& p, const Workspace& ws, hipStream_t s);
// Whether the cooperative K-means with coop_q queries per block should form
// the centroid sums itself: its grid covers every compute unit.
int coop_fused_sums(const Problem& p, int coop_q);
// K-means driver for a problem: 1 one workgroup per unit, 2 one launch pair
// per round, 3 cooperative.
int kmeans_driver(const Problem& p);
// Queries per block of the cooperative K-means for p with at most max_blocks
// blocks per unit, or 0 when its grid does not fit on the device.
int coop_block_queries(const Problem& p, int max_blocks);
hipError_t launch_load_assign(const Problem& p, const int32_t* assign_in, const Workspace& ws,
                              hipStream_t s);
hipError_t launch_csr(const Problem& p, const int32_t* assign, const Workspace& ws, hipStream_t s);
hipError_t launch_centroids(const Problem& p, const Workspace& ws, hipStream_t s);
// Centroid attention: softmax statistics and values; clustered in one key
// chunk also the output rows (otherwise launch_broadcast writes them);
// improved: top-k, mass and rest part (launch_sparse then writes the rows).
// part 0 launches the tile kernel, part 1 the merge of several key chunks
// (nothing for one chunk).
hipError_t launch_centroid_attention(const Problem& p, const Workspace& ws, const int32_t* topk_in,
                                     int part, hipStream_t s);
hipError_t launch_sparse(const Problem& p, const Workspace& ws, hipStream_t s);
hipError_t launch_broadcast(const Problem& p, const int32_t* assign, const Workspace& ws,
                            hipStream_t s);
hipError_t launch_pad_zero(const Problem& p, hipStream_t s);

// Backward pass: scratch buffers carved from the caller's backward workspace.
struct BwdWorkspace {
  float* G;         // [U][C][d]   sum of the members' output gradients
  float* delta;     // [U][C]
  float* dm;        // [U][C]      gradient of the mass (improved)
  float* dqc_part;  // [U][nkb][C][d] centroid-gradient partials per key block
  float* dqc;       // [U][C][d]
  float* part_k;    // [U][C*k][d] key-gradient partials of the top-k rows (improved), key order
  float* part_v;    // [U][C*k][d]
  int32_t* icnt;    // [U][n]      inverse index of the top-k sets: entries per key
  int32_t* ioff;    // [U][n]      first slot of each key in the unit's key-ordered list
  int32_t* epos;    // [U][C*k]    slot of entry (j, r)
};
struct BwdProblem {
  int batch, heads, n, d, dtype, C, topk;  // topk = 0 for the clustered variant
  const void* q;
  const void* k;
  const void* v;
  const void* dout;
  const int32_t* lengths;
  const Workspace* fws;  // the forward pass's state
  BwdWorkspace bws;
  float* dq;
  float* dk;
  float* dv;
};
int bwd_key_blocks(int n);
size_t carve_bwd_workspace(const BwdProblem& p, void* base, BwdWorkspace* ws);
// ev_start / ev_stop (may be null) are recorded around bwd_tile_kernel.
hipError_t launch_backward(const BwdProblem& p, hipStream_t s, hipEvent_t ev_start, hipEvent_t ev_stop);

// Which K-means path runs: 0 automatic, 1 one workgroup per unit, 2 one
// launch pair per round, 3 cooperative (4 / 5: with the centroid sums always
// in the K-means kernel / always in a separate kernel).
void set_kmeans_path(int path);
int kmeans_uses_lds(const Problem& p);

}  // namespace ca
