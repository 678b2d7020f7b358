// C ABI of the library: argument validation, workspace carving and the
// launch sequence of the forward pass on the caller's stream.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <string>

#include "../../include/clustered_attn.h"
#include "kernels.h"

namespace ca {

static thread_local std::string g_last_error;

static int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
static int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

// One-shot event pair around one kernel of the next forward call on this thread.
static thread_local int g_ev_kernel = 0;
static thread_local hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;

static hipError_t mark(int kernel_id, bool start, hipStream_t s) {
  if (g_ev_kernel != kernel_id) return hipSuccess;
  return hipEventRecord(start ? g_ev_start : g_ev_stop, s);
}

static size_t align_up(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

size_t carve_workspace(const Problem& p, void* base, Workspace* ws) {
  const size_t U = static_cast<size_t>(p.units());
  const size_t N = static_cast<size_t>(p.n);
  const size_t C = static_cast<size_t>(p.C);
  const size_t D = static_cast<size_t>(p.d);
  const size_t K = static_cast<size_t>(p.topk > 0 ? p.topk : 1);
  Workspace w;
  w.nblk = (p.n + kKmBlockQ - 1) / kKmBlockQ;
  w.ncsr = (p.n + kCsrBlockQ - 1) / kCsrBlockQ;
  w.nchunk = (p.n + kChunk - 1) / kChunk;
  size_t off = 0;
  auto take = [&](size_t bytes) -> void* {
    void* ptr = base ? static_cast<void*>(static_cast<char*>(base) + off) : nullptr;
    off += align_up(bytes);
    return ptr;
  };
  w.codes = static_cast<uint64_t*>(take(U * N * 8));
  w.assign = static_cast<int32_t*>(take(U * N * 4));
  w.members = static_cast<int32_t*>(take(U * N * 4));
  w.offsets = static_cast<int32_t*>(take(U * (C + 1) * 4));
  w.sizes = static_cast<int32_t*>(take(U * C * 4));
  w.cent = static_cast<uint64_t*>(take(2 * U * C * 8));
  w.part = static_cast<uint32_t*>(take(U * w.nblk * C * 32 * 4));
  w.part_sizes = static_cast<int32_t*>(take(U * w.nblk * C * 4));
  w.csr_cnt = static_cast<int32_t*>(take(U * w.ncsr * C * 4));
  w.qc = static_cast<float*>(take(U * C * D * 4));
  w.pm = static_cast<float*>(take(U * C * w.nchunk * 4));
  w.pz = static_cast<float*>(take(U * C * w.nchunk * 4));
  w.pacc = static_cast<float*>(take(U * C * w.nchunk * D * 4));
  w.cand_idx = static_cast<int32_t*>(take(p.topk > 0 ? U * C * w.nchunk * K * 4 : 0));
  w.cand_val = static_cast<float*>(take(p.topk > 0 ? U * C * w.nchunk * K * 4 : 0));
  w.topk = static_cast<int32_t*>(take(p.topk > 0 ? U * C * K * 4 : 0));
  w.mass = static_cast<float*>(take(p.topk > 0 ? U * C * 4 : 0));
  w.vcb = static_cast<float*>(take(U * C * D * 4));
  w.stats = static_cast<float*>(take(U * C * 2 * 4));
  w.ncoop = coop_max_blocks(p.n, p.units());
  w.coop_q = 0;
  w.coop_sums = 0;
  const size_t NC = static_cast<size_t>(w.ncoop);
  w.sync = static_cast<int32_t*>(take(U * kSyncInts * 4));
  w.ctab = static_cast<uint64_t*>(take(2 * U * static_cast<size_t>(coop_table_stride(p.C)) * 8));
  w.cbases = static_cast<int32_t*>(take(U * NC * C * 4));
  w.clsizes = static_cast<int32_t*>(take(U * NC * C * 4));
  w.qc_part = static_cast<double*>(take(U * C * NC * D * 8));
  w.planes = static_cast<float*>(take(static_cast<size_t>(p.heads) * p.n_bits * D * 4));
  if (ws) *ws = w;
  return off;
}

size_t carve_bwd_workspace(const BwdProblem& p, void* base, BwdWorkspace* ws) {
  const size_t U = static_cast<size_t>(p.batch) * p.heads;
  const size_t N = static_cast<size_t>(p.n);
  const size_t C = static_cast<size_t>(p.C);
  const size_t D = static_cast<size_t>(p.d);
  const size_t K = static_cast<size_t>(p.topk > 0 ? p.topk : 1);
  const size_t nkb = static_cast<size_t>(bwd_key_blocks(p.n));
  const bool improved = p.topk > 0;
  BwdWorkspace w;
  size_t off = 0;
  auto take = [&](size_t bytes) -> void* {
    void* ptr = base ? static_cast<void*>(static_cast<char*>(base) + off) : nullptr;
    off += align_up(bytes);
    return ptr;
  };
  w.G = static_cast<float*>(take(U * C * D * 4));
  w.delta = static_cast<float*>(take(U * C * 4));
  w.dm = static_cast<float*>(take(U * C * 4));
  w.dqc_part = static_cast<float*>(take(U * nkb * C * D * 4));
  w.dqc = static_cast<float*>(take(U * C * D * 4));
  w.part_k = static_cast<float*>(take(improved ? U * C * K * D * 4 : 0));
  w.part_v = static_cast<float*>(take(improved ? U * C * K * D * 4 : 0));
  w.icnt = static_cast<int32_t*>(take(improved ? U * N * 4 : 0));
  w.ioff = static_cast<int32_t*>(take(improved ? U * N * 4 : 0));
  w.epos = static_cast<int32_t*>(take(improved ? U * C * K * 4 : 0));
  if (ws) *ws = w;
  return off;
}

size_t carve_otop_workspace(const Problem& p, void* base, Workspace* ws) {
  const size_t U = static_cast<size_t>(p.units());
  const size_t N = static_cast<size_t>(p.n);
  const size_t K = static_cast<size_t>(p.topk > 0 ? p.topk : 1);
  Workspace w{};
  w.nchunk = (p.n + kChunk - 1) / kChunk;
  size_t off = 0;
  auto take = [&](size_t bytes) -> void* {
    void* ptr = base ? static_cast<void*>(static_cast<char*>(base) + off) : nullptr;
    off += align_up(bytes);
    return ptr;
  };
  w.topk = static_cast<int32_t*>(take(U * N * K * 4));
  if (w.nchunk > 1) {
    w.cand_idx = static_cast<int32_t*>(take(U * N * w.nchunk * K * 4));
    w.cand_val = static_cast<float*>(take(U * N * w.nchunk * K * 4));
  }
  if (ws) *ws = w;
  return off;
}

// Returns CA_OK or an error code (message recorded) for the given sizes.
static int check_sizes(int batch, int heads, int n, int d, int dtype, int C, int n_bits, int L,
                       int topk, bool improved) {
  if (batch < 1 || heads < 1 || n < 1 || d < 1)
    return fail(CA_ERR_INVALID_ARG, "batch, heads, n and d must be >= 1 (got %d, %d, %d, %d)",
                batch, heads, n, d);
  if (dtype != CA_F32 && dtype != CA_BF16)
    return fail(CA_ERR_INVALID_ARG, "dtype must be CA_F32 or CA_BF16 (got %d)", dtype);
  if (n_bits < 1) return fail(CA_ERR_INVALID_ARG, "n_bits must be >= 1 (got %d)", n_bits);
  if (C < 1) return fail(CA_ERR_INVALID_ARG, "n_clusters must be >= 1 (got %d)", C);
  if (L < 1) return fail(CA_ERR_INVALID_ARG, "lloyd_iters must be >= 1 (got %d)", L);
  if (improved && topk < 1) return fail(CA_ERR_INVALID_ARG, "topk must be >= 1 (got %d)", topk);
  if (d != 32 && d != 64) return fail(CA_ERR_UNSUPPORTED, "d must be 32 or 64 (got %d)", d);
  if (n_bits > 64) return fail(CA_ERR_UNSUPPORTED, "n_bits must be <= 64 (got %d)", n_bits);
  if (C > 256) return fail(CA_ERR_UNSUPPORTED, "n_clusters must be <= 256 (got %d)", C);
  if (L > 1000) return fail(CA_ERR_UNSUPPORTED, "lloyd_iters must be <= 1000 (got %d)", L);
  if (improved && topk > 128) return fail(CA_ERR_UNSUPPORTED, "topk must be <= 128 (got %d)", topk);
  if (n > (1 << 20)) return fail(CA_ERR_UNSUPPORTED, "n must be <= 1048576 (got %d)", n);
  const long long rows = static_cast<long long>(batch) * heads * n;
  if (rows >= (1ll << 31)) return fail(CA_ERR_UNSUPPORTED, "batch*heads*n must be < 2^31");
  if (static_cast<long long>(batch) * heads > 65535)
    return fail(CA_ERR_UNSUPPORTED, "batch*heads must be <= 65535");
  return CA_OK;
}

static int run_forward(const void* q, const void* k, const void* v, const int32_t* lengths,
                       const float* planes, int batch, int heads, int n, int d, int dtype, int C,
                       int n_bits, int L, uint64_t seed, int topk, void* out, void* workspace,
                       size_t workspace_bytes, const ca_aux* aux, void* stream) {
  const bool improved = topk > 0;
  int rc = check_sizes(batch, heads, n, d, dtype, C, n_bits, L, topk, improved);
  if (rc != CA_OK) return rc;
  const bool assign_given = aux && aux->assign_in;
  if (!q || !k || !v || !out)
    return fail(CA_ERR_INVALID_ARG, "q, k, v and out must not be NULL");
  Problem p;
  p.batch = batch;
  p.heads = heads;
  p.n = n;
  p.d = d;
  p.dtype = dtype;
  p.C = C;
  p.n_bits = n_bits;
  p.L = L;
  p.topk = improved ? topk : 0;
  p.q = q;
  p.k = k;
  p.v = v;
  p.lengths = lengths;
  p.planes = planes;
  p.out = out;
  const size_t need = carve_workspace(p, nullptr, nullptr);
  if (!workspace) return fail(CA_ERR_WORKSPACE, "workspace must not be NULL (%zu bytes needed)", need);
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(CA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < need)
    return fail(CA_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, need);
  Workspace ws;
  carve_workspace(p, workspace, &ws);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // launch errors are read with hipGetLastError after each launch: drop a
  // stale error left by an earlier, unrelated runtime call of this thread
  (void)hipGetLastError();

  hipError_t e = hipSuccess;
#define CA_TRY(call)                                                                  \
  do {                                                                                \
    e = (call);                                                                       \
    if (e != hipSuccess)                                                              \
      return fail(CA_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e));          \
  } while (0)

  const uint64_t* codes_in = aux ? aux->codes_in : nullptr;
  const int driver = kmeans_driver(p);
  if (!planes) {  // drawn from the seed before anything hashes (outside the timed stages)
    CA_TRY(launch_planes(p, seed, ws.planes, s));
    p.planes = ws.planes;
  }
  if (assign_given) {
    CA_TRY(launch_load_assign(p, aux->assign_in, ws, s));
    CA_TRY(mark(CA_KERNEL_CENTROIDS, true, s));
    CA_TRY(launch_csr(p, ws.assign, ws, s));
    CA_TRY(launch_centroids(p, ws, s));
    CA_TRY(mark(CA_KERNEL_CENTROIDS, false, s));
  } else if (driver == 1) {
    // one kernel: hashing, K-means, member lists and centroids
    CA_TRY(mark(CA_KERNEL_KMEANS, true, s));
    CA_TRY(launch_cluster_lds(p, codes_in, ws, s));
    CA_TRY(mark(CA_KERNEL_KMEANS, false, s));
  } else {
    if (codes_in) {
      CA_TRY(launch_load_codes(p, codes_in, ws, s));
    } else {
      CA_TRY(mark(CA_KERNEL_HASH, true, s));
      CA_TRY(launch_hash(p, ws, s));
      CA_TRY(mark(CA_KERNEL_HASH, false, s));
    }
    if (driver == 3) {
      // all rounds and the member lists in one launch
      ws.coop_q = coop_block_queries(p, ws.ncoop);
      ws.coop_sums = coop_fused_sums(p, ws.coop_q);
      CA_TRY(mark(CA_KERNEL_KMEANS, true, s));
      CA_TRY(launch_kmeans_coop(p, ws, s));
      CA_TRY(mark(CA_KERNEL_KMEANS, false, s));
      CA_TRY(mark(CA_KERNEL_CENTROIDS, true, s));
      CA_TRY(launch_coop_centroids(p, ws, s));
      CA_TRY(mark(CA_KERNEL_CENTROIDS, false, s));
    } else {
      CA_TRY(mark(CA_KERNEL_KMEANS, true, s));
      CA_TRY(launch_kmeans(p, ws, s));
      CA_TRY(mark(CA_KERNEL_KMEANS, false, s));
      CA_TRY(mark(CA_KERNEL_CENTROIDS, true, s));
      CA_TRY(launch_csr(p, ws.assign, ws, s));
      CA_TRY(launch_centroids(p, ws, s));
      CA_TRY(mark(CA_KERNEL_CENTROIDS, false, s));
    }
  }
  CA_TRY(mark(CA_KERNEL_CENTROID_ATTN, true, s));
  CA_TRY(mark(CA_KERNEL_ATTN_TILE, true, s));
  CA_TRY(launch_centroid_attention(p, ws, improved && aux ? aux->topk_in : nullptr, 0, s));
  CA_TRY(mark(CA_KERNEL_ATTN_TILE, false, s));
  CA_TRY(launch_centroid_attention(p, ws, improved && aux ? aux->topk_in : nullptr, 1, s));
  CA_TRY(mark(CA_KERNEL_CENTROID_ATTN, false, s));
  CA_TRY(mark(CA_KERNEL_OUTPUT, true, s));
  if (improved) CA_TRY(launch_sparse(p, ws, s));
  if (!improved && ws.nchunk > 1) {
    CA_TRY(launch_broadcast(p, ws.assign, ws, s));  // also zeroes the padded rows
  } else if (lengths && (assign_given || (codes_in && driver != 1))) {
    CA_TRY(launch_pad_zero(p, s));  // otherwise the hashing or clustering kernel zeroed them
  }
  CA_TRY(mark(CA_KERNEL_OUTPUT, false, s));
  g_ev_kernel = 0;
  if (aux) {
    const size_t U = static_cast<size_t>(batch) * heads;
    auto copy = [&](void* dst, const void* src, size_t bytes) -> hipError_t {
      if (!dst) return hipSuccess;
      return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, s);
    };
    if (!assign_given) CA_TRY(copy(aux->codes_out, ws.codes, U * n * 8));
    CA_TRY(copy(aux->assign_out, ws.assign, U * n * 4));
    CA_TRY(copy(aux->sizes_out, ws.sizes, U * C * 4));
    CA_TRY(copy(aux->centroids_out, ws.qc, U * C * d * 4));
    CA_TRY(copy(aux->values_out, ws.vcb, U * C * d * 4));
    if (improved) {
      CA_TRY(copy(aux->topk_out, ws.topk, U * C * topk * 4));
      CA_TRY(copy(aux->mass_out, ws.mass, U * C * 4));
    }
    CA_TRY(copy(aux->planes_out, p.planes, static_cast<size_t>(heads) * n_bits * d * 4));
  }
#undef CA_TRY
  return CA_OK;
}

static int run_oracle_top(const void* q, const void* k, const void* v, const int32_t* lengths,
                          int batch, int heads, int n, int d, int dtype, int topk, void* out,
                          int32_t* topk_out, void* workspace, size_t workspace_bytes,
                          void* stream) {
  int rc = check_sizes(batch, heads, n, d, dtype, 1, 1, 1, topk, true);
  if (rc != CA_OK) return rc;
  if (!q || !k || !v || !out) return fail(CA_ERR_INVALID_ARG, "q, k, v and out must not be NULL");
  Problem p;
  memset(&p, 0, sizeof(p));
  p.batch = batch;
  p.heads = heads;
  p.n = n;
  p.d = d;
  p.dtype = dtype;
  p.C = n;  // one row per query
  p.topk = topk;
  p.q = q;
  p.k = k;
  p.v = v;
  p.lengths = lengths;
  p.out = out;
  const size_t need = carve_otop_workspace(p, nullptr, nullptr);
  if (!workspace) return fail(CA_ERR_WORKSPACE, "workspace must not be NULL (%zu bytes needed)", need);
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(CA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < need)
    return fail(CA_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, need);
  Workspace ws;
  carve_otop_workspace(p, workspace, &ws);
  if (topk_out) ws.topk = topk_out;  // the kernels write the sets in place
  hipStream_t s = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  hipError_t e = mark(CA_KERNEL_CENTROID_ATTN, true, s);
  if (e == hipSuccess) e = launch_oracle_top(p, ws, s);
  if (e == hipSuccess) e = mark(CA_KERNEL_CENTROID_ATTN, false, s);
  g_ev_kernel = 0;
  if (e != hipSuccess) return fail(CA_ERR_HIP, "oracle-top launch failed: %s", hipGetErrorString(e));
  return CA_OK;
}

static int run_backward(const void* q, const void* k, const void* v, const int32_t* lengths,
                        int batch, int heads, int n, int d, int dtype, int C, int topk,
                        const void* dout, float* dq, float* dk, float* dv, const void* workspace,
                        size_t workspace_bytes, void* bwd_workspace, size_t bwd_workspace_bytes,
                        void* stream) {
  const bool improved = topk > 0;
  int rc = check_sizes(batch, heads, n, d, dtype, C, 1, 1, topk, improved);
  if (rc != CA_OK) return rc;
  if (!q || !k || !v || !dout || !dq || !dk || !dv)
    return fail(CA_ERR_INVALID_ARG, "q, k, v, dout, dq, dk and dv must not be NULL");
  Problem p;
  memset(&p, 0, sizeof(p));
  p.batch = batch;
  p.heads = heads;
  p.n = n;
  p.d = d;
  p.dtype = dtype;
  p.C = C;
  p.n_bits = 1;
  p.L = 1;
  p.topk = improved ? topk : 0;
  const size_t need = carve_workspace(p, nullptr, nullptr);
  if (!workspace) return fail(CA_ERR_WORKSPACE, "workspace (the forward pass's) must not be NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(CA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (workspace_bytes < need)
    return fail(CA_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, need);
  Workspace fws;
  carve_workspace(p, const_cast<void*>(workspace), &fws);
  BwdProblem b;
  b.batch = batch;
  b.heads = heads;
  b.n = n;
  b.d = d;
  b.dtype = dtype;
  b.C = C;
  b.topk = p.topk;
  b.q = q;
  b.k = k;
  b.v = v;
  b.dout = dout;
  b.lengths = lengths;
  b.fws = &fws;
  b.dq = dq;
  b.dk = dk;
  b.dv = dv;
  const size_t bneed = carve_bwd_workspace(b, nullptr, nullptr);
  if (!bwd_workspace) return fail(CA_ERR_WORKSPACE, "bwd_workspace must not be NULL (%zu bytes needed)", bneed);
  if (reinterpret_cast<uintptr_t>(bwd_workspace) % 256 != 0)
    return fail(CA_ERR_WORKSPACE, "bwd_workspace must be 256-byte aligned");
  if (bwd_workspace_bytes < bneed)
    return fail(CA_ERR_WORKSPACE, "bwd_workspace too small: %zu bytes given, %zu needed",
                bwd_workspace_bytes, bneed);
  carve_bwd_workspace(b, bwd_workspace, &b.bws);
  (void)hipGetLastError();
  const bool timed = g_ev_kernel == CA_KERNEL_BWD_CENTROID;
  const hipError_t e = launch_backward(b, static_cast<hipStream_t>(stream), timed ? g_ev_start : nullptr,
                                       timed ? g_ev_stop : nullptr);
  if (timed) g_ev_kernel = 0;
  if (e != hipSuccess) return fail(CA_ERR_HIP, "backward launch failed: %s", hipGetErrorString(e));
  return CA_OK;
}

// Device-resident scratch of the allocation-free entry point: one array per
// GPU that the library runs on, held until the process ends, shared by every
// call on that GPU.  Host code never uses the array's name as an address: its
// device address comes from hipGetSymbolAddress once per device.
constexpr size_t kScratchBytes = static_cast<size_t>(CA_NOALLOC_SCRATCH_BYTES);
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
static void* g_scratch_ptr[kMaxDevices] = {nullptr};
static std::mutex g_scratch_mutex;

// The current device's scratch address, looked up on its first use (with that
// device current); null with the error recorded if the lookup fails.
static void* scratch_address(int* rc) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *rc = fail(CA_ERR_HIP, "hipGetDevice failed or device index out of range: %s", hipGetErrorString(e));
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr) {
      *rc = fail(CA_ERR_HIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                 hipGetErrorString(e));
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  *rc = CA_OK;
  return g_scratch_ptr[dev];
}

}  // namespace ca

extern "C" {

size_t ca_workspace_bytes(int batch, int heads, int n, int d, int dtype, int n_clusters,
                          int n_bits, int topk) {
  const bool improved = topk > 0;
  if (ca::check_sizes(batch, heads, n, d, dtype, n_clusters, n_bits, 1, topk, improved) != CA_OK)
    return 0;
  ca::Problem p;
  memset(&p, 0, sizeof(p));
  p.batch = batch;
  p.heads = heads;
  p.n = n;
  p.d = d;
  p.dtype = dtype;
  p.C = n_clusters;
  p.n_bits = n_bits;
  p.L = 1;
  p.topk = improved ? topk : 0;
  return ca::carve_workspace(p, nullptr, nullptr);
}

int clustered_attention_fwd(const void* q, const void* k, const void* v, const int32_t* lengths,
                            const float* planes, int batch, int heads, int n, int d, int dtype,
                            int n_clusters, int n_bits, int lloyd_iters, uint64_t seed, void* out,
                            void* workspace, size_t workspace_bytes, const ca_aux* aux,
                            void* stream) {
  try {
    return ca::run_forward(q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters,
                           n_bits, lloyd_iters, seed, 0, out, workspace, workspace_bytes, aux,
                           stream);
  } catch (...) {
    return ca::fail(CA_ERR_HIP, "unexpected C++ exception");
  }
}

int iclustered_attention_fwd(const void* q, const void* k, const void* v, const int32_t* lengths,
                             const float* planes, int batch, int heads, int n, int d, int dtype,
                             int n_clusters, int n_bits, int lloyd_iters, uint64_t seed, int topk,
                             void* out, void* workspace, size_t workspace_bytes,
                             const ca_aux* aux, void* stream) {
  try {
    if (topk < 1) return ca::fail(CA_ERR_INVALID_ARG, "topk must be >= 1 (got %d)", topk);
    return ca::run_forward(q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters,
                           n_bits, lloyd_iters, seed, topk, out, workspace, workspace_bytes, aux,
                           stream);
  } catch (...) {
    return ca::fail(CA_ERR_HIP, "unexpected C++ exception");
  }
}

int iclustered_attention_fwd_noalloc(const void* q, const void* k, const void* v,
                                     const int32_t* lengths, const float* planes, int batch,
                                     int heads, int n, int d, int dtype, int n_clusters,
                                     int n_bits, int lloyd_iters, uint64_t seed, int topk,
                                     void* out, const ca_aux* aux, void* stream) {
  try {
    if (topk < 1) return ca::fail(CA_ERR_INVALID_ARG, "topk must be >= 1 (got %d)", topk);
    // sizes first, so that a rejected call touches no device state
    const size_t need = ca_workspace_bytes(batch, heads, n, d, dtype, n_clusters, n_bits, topk);
    if (need == 0)
      return ca::run_forward(q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters,
                             n_bits, lloyd_iters, seed, topk, out, nullptr, 0, aux, stream);
    if (need > ca::kScratchBytes)
      return ca::fail(CA_ERR_UNSUPPORTED,
                      "these sizes need %zu bytes of scratch; the allocation-free entry point holds %zu",
                      need, ca::kScratchBytes);
    int rc = CA_OK;
    void* ws = ca::scratch_address(&rc);
    if (ws == nullptr) return rc;
    return ca::run_forward(q, k, v, lengths, planes, batch, heads, n, d, dtype, n_clusters, n_bits,
                           lloyd_iters, seed, topk, out, ws, ca::kScratchBytes, aux, stream);
  } catch (...) {
    return ca::fail(CA_ERR_HIP, "unexpected C++ exception");
  }
}

size_t ca_backward_workspace_bytes(int batch, int heads, int n, int d, int dtype, int n_clusters,
                                   int topk) {
  const bool improved = topk > 0;
  if (ca::check_sizes(batch, heads, n, d, dtype, n_clusters, 1, 1, topk, improved) != CA_OK) return 0;
  ca::BwdProblem b;
  memset(&b, 0, sizeof(b));
  b.batch = batch;
  b.heads = heads;
  b.n = n;
  b.d = d;
  b.dtype = dtype;
  b.C = n_clusters;
  b.topk = improved ? topk : 0;
  return ca::carve_bwd_workspace(b, nullptr, nullptr);
}

int clustered_attention_bwd(const void* q, const void* k, const void* v, const int32_t* lengths,
                            int batch, int heads, int n, int d, int dtype, int n_clusters,
                            const void* dout, float* dq, float* dk, float* dv,
                            const void* workspace, size_t workspace_bytes, void* bwd_workspace,
                            size_t bwd_workspace_bytes, void* stream) {
  try {
    return ca::run_backward(q, k, v, lengths, batch, heads, n, d, dtype, n_clusters, 0, dout, dq,
                            dk, dv, workspace, workspace_bytes, bwd_workspace,
                            bwd_workspace_bytes, stream);
  } catch (...) {
    return ca::fail(CA_ERR_HIP, "unexpected C++ exception");
  }
}

int iclustered_attention_bwd(const void* q, const void* k, const void* v, const int32_t* lengths,
                             int batch, int heads, int n, int d, int dtype, int n_clusters,
                             int topk, const void* dout, float* dq, float* dk, float* dv,
                             const void* workspace, size_t workspace_bytes, void* bwd_workspace,
                             size_t bwd_workspace_bytes, void* stream) {
  try {
    if (topk < 1) return ca::fail(CA_ERR_INVALID_ARG, "topk must be >= 1 (got %d)", topk);
    return ca::run_backward(q, k, v, lengths, batch, heads, n, d, dtype, n_clusters, topk, dout,
                            dq, dk, dv, workspace, workspace_bytes, bwd_workspace,
                            bwd_workspace_bytes, stream);
  } catch (...) {
    return ca::fail(CA_ERR_HIP, "unexpected C++ exception");
  }
}

size_t ca_oracle_top_workspace_bytes(int batch, int heads, int n, int d, int dtype, int topk) {
  if (ca::check_sizes(batch, heads, n, d, dtype, 1, 1, 1, topk, true) != CA_OK) return 0;
  ca::Problem p;
  memset(&p, 0, sizeof(p));
  p.batch = batch;
  p.heads = heads;
  p.n = n;
  p.d = d;
  p.dtype = dtype;
  p.C = n;
  p.topk = topk;
  return ca::carve_otop_workspace(p, nullptr, nullptr);
}

int oracle_top_attention_fwd(const void* q, const void* k, const void* v, const int32_t* lengths,
                             int batch, int heads, int n, int d, int dtype, int topk, void* out,
                             int32_t* topk_out, void* workspace, size_t workspace_bytes,
                             void* stream) {
  try {
    if (topk < 1) return ca::fail(CA_ERR_INVALID_ARG, "topk must be >= 1 (got %d)", topk);
    return ca::run_oracle_top(q, k, v, lengths, batch, heads, n, d, dtype, topk, out, topk_out,
                              workspace, workspace_bytes, stream);
  } catch (...) {
    return ca::fail(CA_ERR_HIP, "unexpected C++ exception");
  }
}

const char* ca_last_error(void) { return ca::g_last_error.c_str(); }

int ca_version(void) { return 200; }

int ca_time_next_stage(int stage, void* start_event, void* stop_event) {
  if (stage < 0 || stage > CA_KERNEL_ATTN_TILE || (stage != 0 && (!start_event || !stop_event)))
    return ca::fail(CA_ERR_INVALID_ARG, "invalid stage %d or null event", stage);
  ca::g_ev_kernel = stage;
  ca::g_ev_start = static_cast<hipEvent_t>(start_event);
  ca::g_ev_stop = static_cast<hipEvent_t>(stop_event);
  return CA_OK;
}

// Selects the K-means driver (0 automatic, 1 one workgroup per unit, 2 one
// launch pair per round, 3 cooperative; 4 and 5 cooperative with the centroid
// sums formed by the K-means kernel or by a separate kernel).  Exposed for
// tests that cover every driver.
int ca_set_kmeans_path(int path) {
  if (path < 0 || path > 5) return ca::fail(CA_ERR_INVALID_ARG, "path must be 0 to 5");
  ca::set_kmeans_path(path);
  return CA_OK;
}

}  // extern "C"
