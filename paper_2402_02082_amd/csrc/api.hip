// C ABI of libglide: argument checking, workspace planning and launches.
// Every check that does not need device data runs before any HIP call, so
// the error paths are testable on a machine without a GPU.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "glide.h"
#include "internal.h"

// Fixed scratch of glide_tree_attn_noalloc (see scratch_of_current_device).
static constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace {

thread_local int g_last_hip_error = 0;

int hip_status(hipError_t e) {
  if (e == hipSuccess) return GLIDE_OK;
  g_last_hip_error = (int)e;
  return GLIDE_EHIP;
}

bool validate_enabled() {
  const char* v = getenv("GLIDE_VALIDATE");
  return v && v[0] && strcmp(v, "0") != 0;
}

// Copies a small int32 device array to the host (synchronises `stream`).
bool fetch_ints(const int32_t* dev, size_t n, std::vector<int32_t>& host, hipStream_t stream,
                int* status) {
  host.resize(n);
  hipError_t e = hipMemcpyAsync(host.data(), dev, n * sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) {
    *status = hip_status(e);
    return false;
  }
  return true;
}

bool parents_ok(const std::vector<int32_t>& parents, int B, int N) {
  for (int b = 0; b < B; ++b)
    for (int n = 0; n < N; ++n) {
      const int p = parents[(size_t)b * N + n];
      if (p < -1 || p >= n) return false;
    }
  return true;
}

// Kernels keep key-row byte offsets inside one (sequence, head) slab in
// 32-bit registers (buffer descriptors: rows * 512 bytes for float32), and
// the split merge counts its output rows B * N * H in an int.
constexpr int kMaxKeys = 1 << 22;

bool tree_attn_sizes_ok(int B, int N, int H, int D, int L_cap, bool tree) {
  if (B < 1 || B > 65535 || H < 1 || N < 1 || N > glide::kMaxNodes) return false;  // B is a grid dim
  if (D != glide::kHeadDim) return false;
  if (L_cap < (tree ? N : 1) || L_cap > kMaxKeys) return false;
  if ((double)B * N * H > 2147483647.0) return false;
  // keep every element offset inside size_t
  if ((double)B * H * (double)L_cap * D > 9.0e18) return false;
  return true;
}

glide::AttnArgs attn_args(const void* q, const void* k_cache, const void* v_cache,
                          const int32_t* seq_lens, const int32_t* tree_parents, void* out, int B,
                          int N, int H, int D, int L_cap, float scale, const glide::AttnPlan& plan,
                          void* workspace) {
  glide::AttnArgs a{};
  a.q = q;
  a.k = k_cache;
  a.v = v_cache;
  a.seq_lens = seq_lens;
  a.parents = tree_parents;
  a.out = out;
  char* ws = (char*)workspace;
  a.part_o = plan.ws_bytes ? (float*)(ws + plan.part_o_off) : nullptr;
  a.part_ml = plan.ws_bytes ? (float2*)(ws + plan.part_ml_off) : nullptr;
  a.counters = plan.ws_bytes && plan.merge_in_kernel ? (unsigned*)(ws + plan.counters_off) : nullptr;
  a.part_h = plan.ws_bytes && plan.half_states ? (uint16_t*)(ws + plan.part_h_off) : nullptr;
  a.B = B;
  a.N = N;
  a.H = H;
  a.L_cap = L_cap;
  a.chunk = plan.chunk;
  a.splits = plan.splits;
  const double sc = scale > 0.f ? (double)scale : 1.0 / sqrt((double)D);
  a.scale_log2 = (float)(sc * 1.4426950408889634);  // log2(e)
  return a;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

bool rows_matmul_sizes_ok(int M, int K, int N) {
  return M >= 1 && N >= 1 && K >= 8 && K % 8 == 0 && K <= glide::kMaxMatmulK;
}

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// CaPE's part kernel runs one workgroup row per draft row: B * gamma is a
// grid dimension (at most 65535).
bool cape_rows_ok(int B, int gamma) { return (long)B * gamma <= 65535; }

// Workspace of the cross-attention block: the attention's split workspace
// first (so its arrival counters sit at offset 0 whatever the shape), then
// the projected queries and the concatenated heads (both bf16 [B, Nq, H, D]).
struct CrossPlan {
  glide::AttnPlan attn;
  size_t q_off, heads_off, attn_off, bytes;
};

bool cross_block_plan(int B, int Nq, int d_D, int H, int D, int L_cap, CrossPlan* p) {
  if (!tree_attn_sizes_ok(B, Nq, H, D, L_cap, false)) return false;
  if (!rows_matmul_sizes_ok(B * Nq, d_D, H * D) || (double)B * Nq > 1.0e9) return false;
  p->attn = glide::plan_tree_attn(B, Nq, H, L_cap, 0);
  const size_t rows = align256((size_t)B * Nq * H * D * 2);
  p->attn_off = 0;
  p->q_off = align256(p->attn.ws_bytes);
  p->heads_off = p->q_off + rows;
  p->bytes = p->heads_off + rows;
  return true;
}

// ---------------------------------------------------------------------------
// Fixed scratch of glide_tree_attn_noalloc, for callers that cannot allocate:
// a file-scope device array that every GPU the library runs on holds until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// the device memory, so its device address is looked up once per device
// (with that device current) and only that address is used from then on.
// ---------------------------------------------------------------------------
constexpr int kMaxDevices = 64;


std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

int scratch_of_current_device(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e);
  if (dev < 0 || dev >= kMaxDevices) return GLIDE_EINVAL;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e);
    if (!p) return hip_status(hipErrorInvalidSymbol);
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return GLIDE_OK;
}


// Shared body of glide_tree_attn and glide_tree_attn_noalloc.  With
// `scratch` set, the split partials go to the per-device scratch array that
// it resolves (after every host-side check) instead of the caller's
// workspace, and plans that need more than that array holds are refused.
int tree_attn_call(const void* q, const void* k_cache, const void* v_cache, const int32_t* seq_lens,
                   const int32_t* tree_parents, void* out, int B, int N, int H, int D, int L_cap,
                   int dtype, float scale, int max_splits, void* workspace, size_t ws_bytes,
                   int (*scratch)(void** ptr), hipStream_t stream) {
  const bool tree = tree_parents != nullptr;
  if (!q || !k_cache || !v_cache || !seq_lens || !out) return GLIDE_EINVAL;
  if (dtype != GLIDE_BF16 && dtype != GLIDE_F32) return GLIDE_EINVAL;
  if (!tree_attn_sizes_ok(B, N, H, D, L_cap, tree)) return GLIDE_EINVAL;
  if (max_splits < 0 || max_splits > glide::kMaxSplits) return GLIDE_EINVAL;
  if (!isfinite(scale)) return GLIDE_EINVAL;
  const glide::AttnPlan plan = glide::plan_tree_attn(B, N, H, L_cap, max_splits);
  if (scratch) {
    if (plan.ws_bytes > kNoAllocScratchBytes) return GLIDE_ESCRATCH;
    if (plan.ws_bytes > 0) {
      const int st = scratch(&workspace);
      if (st != GLIDE_OK) return st;
      ws_bytes = kNoAllocScratchBytes;
    }
  }
  if (plan.ws_bytes > 0 && (!workspace || ws_bytes < plan.ws_bytes)) return GLIDE_EINVAL;

  if (validate_enabled()) {
    int status = GLIDE_OK;
    std::vector<int32_t> lens, par;
    if (!fetch_ints(seq_lens, (size_t)B, lens, stream, &status)) return status;
    for (int b = 0; b < B; ++b)
      if (lens[b] < 0 || lens[b] > L_cap - (tree ? N : 0)) return GLIDE_ERANGE;
    if (tree) {
      if (!fetch_ints(tree_parents, (size_t)B * N, par, stream, &status)) return status;
      if (!parents_ok(par, B, N)) return GLIDE_ERANGE;
    }
  }

  const glide::AttnArgs a = attn_args(q, k_cache, v_cache, seq_lens, tree_parents, out, B, N, H, D,
                                      L_cap, scale, plan, workspace);
  return hip_status(glide::launch_tree_attn(a, dtype == GLIDE_BF16, stream));
}


}  // namespace

extern "C" {

const char* glide_strerror(int status) {
  switch (status) {
    case GLIDE_OK: return "ok";
    case GLIDE_EINVAL: return "invalid argument";
    case GLIDE_ERANGE: return "device data out of range";
    case GLIDE_EHIP: return "HIP error";
    case GLIDE_ESCRATCH: return "sizes need more than the fixed scratch of the no-allocation call";
    default: return "unknown status";
  }
}

int glide_last_hip_error(void) { return g_last_hip_error; }

size_t glide_tree_attn_workspace(int B, int N, int H, int D, int L_cap, int max_splits) {
  if (!tree_attn_sizes_ok(B, N, H, D, L_cap, false)) return 0;
  if (max_splits < 0 || max_splits > glide::kMaxSplits) return 0;
  return glide::plan_tree_attn(B, N, H, L_cap, max_splits).ws_bytes;
}

int glide_tree_attn(const void* q, const void* k_cache, const void* v_cache, const int32_t* seq_lens,
                    const int32_t* tree_parents, void* out, int B, int N, int H, int D, int L_cap,
                    int dtype, float scale, int max_splits, void* workspace, size_t ws_bytes,
                    hipStream_t stream) {
  return tree_attn_call(q, k_cache, v_cache, seq_lens, tree_parents, out, B, N, H, D, L_cap, dtype, scale,
                        max_splits, workspace, ws_bytes, nullptr, stream);
}

size_t glide_tree_attn_noalloc_max_workspace(void) { return kNoAllocScratchBytes; }

int glide_tree_attn_noalloc(const void* q, const void* k_cache, const void* v_cache,
                            const int32_t* seq_lens, const int32_t* tree_parents, void* out, int B, int N,
                            int H, int D, int L_cap, int dtype, float scale, int max_splits,
                            hipStream_t stream) {
  return tree_attn_call(q, k_cache, v_cache, seq_lens, tree_parents, out, B, N, H, D, L_cap, dtype, scale,
                        max_splits, nullptr, 0, &scratch_of_current_device, stream);
}

size_t cape_expand_workspace(int B, int gamma, int V) {
  if (B < 1 || gamma < 1 || gamma > glide::kMaxNodes || V < 2 || !cape_rows_ok(B, gamma)) return 0;
  return glide::cape_workspace_bytes(B, gamma, V);
}

int cape_expand(const float* draft_probs, int B, int gamma, int V, int k, int fixed, int n_max,
                int32_t* tokens_out, int32_t* parents_out, int32_t* n_nodes_out, void* workspace,
                size_t ws_bytes, hipStream_t stream) {
  if (!draft_probs || !tokens_out || !parents_out || !n_nodes_out || !workspace) return GLIDE_EINVAL;
  if (B < 1 || gamma < 1 || n_max < gamma || n_max > glide::kMaxNodes || V < 2) return GLIDE_EINVAL;
  if (!cape_rows_ok(B, gamma)) return GLIDE_EINVAL;
  if (k < 0 || (fixed && k > GLIDE_CAPE_MAX_K)) return GLIDE_EINVAL;
  if ((double)B * gamma * V > 9.0e18) return GLIDE_EINVAL;
  if (ws_bytes < glide::cape_workspace_bytes(B, gamma, V)) return GLIDE_EINVAL;
  return hip_status(glide::launch_cape_expand(draft_probs, B, gamma, V, k, fixed ? 1 : 0, n_max,
                                              tokens_out, parents_out, n_nodes_out, workspace,
                                              stream));
}

int glide_argmax_rows(const float* logits, int rows, int V, int32_t* idx_out, hipStream_t stream) {
  if (!logits || !idx_out || rows < 1 || V < 1) return GLIDE_EINVAL;
  if ((double)rows * V > 9.0e18) return GLIDE_EINVAL;
  return hip_status(glide::launch_argmax_rows(logits, rows, V, idx_out, stream));
}

int tree_verify(const int32_t* target_argmax, const int32_t* cand_tokens, const int32_t* parents,
                int B, int N, int32_t* accept_len, int32_t* last_node, int32_t* bonus,
                hipStream_t stream) {
  if (!target_argmax || !cand_tokens || !parents || !accept_len) return GLIDE_EINVAL;
  if (B < 1 || N < 1 || N > glide::kMaxNodes) return GLIDE_EINVAL;
  if (validate_enabled()) {
    int status = GLIDE_OK;
    std::vector<int32_t> par;
    if (!fetch_ints(parents, (size_t)B * N, par, stream, &status)) return status;
    if (!parents_ok(par, B, N)) return GLIDE_ERANGE;
  }
  return hip_status(glide::launch_tree_verify(target_argmax, cand_tokens, parents, B, N, accept_len,
                                              last_node, bonus, stream));
}

int glide_verify_commit(const float* logits, int V, const int32_t* cand_tokens, const int32_t* parents,
                        int B, int N, void* const* k_caches, void* const* v_caches, int layers, int H,
                        int D, int L_cap, int dtype, const int32_t* seq_lens, int32_t* seq_lens_out,
                        int32_t* target_argmax, int32_t* accept_len, int32_t* last_node, int32_t* bonus,
                        int32_t* path, hipStream_t stream) {
  if (!logits || !cand_tokens || !parents || !seq_lens || !seq_lens_out || !target_argmax ||
      !accept_len)
    return GLIDE_EINVAL;
  if (seq_lens_out == seq_lens) return GLIDE_EINVAL;  // other workgroups still read the lengths
  if (V < 1 || B < 1 || B > 65535 || N < 1 || N > glide::kMaxNodes) return GLIDE_EINVAL;
  if ((double)B * (N + 1) * V > 9.0e18) return GLIDE_EINVAL;
  if (layers < 0 || layers > glide::kMaxLayers) return GLIDE_EINVAL;
  if (dtype != GLIDE_BF16 && dtype != GLIDE_F32) return GLIDE_EINVAL;
  if (!tree_attn_sizes_ok(B, N, H, D, L_cap, true)) return GLIDE_EINVAL;
  if (layers > 0 && (!k_caches || !v_caches)) return GLIDE_EINVAL;
  glide::CommitArgs a{};
  for (int l = 0; l < layers; ++l) {
    if (!k_caches[l] || !v_caches[l]) return GLIDE_EINVAL;
    a.k[l] = (char*)k_caches[l];
    a.v[l] = (char*)v_caches[l];
  }
  if (validate_enabled()) {
    int status = GLIDE_OK;
    std::vector<int32_t> lens, par;
    if (layers > 0) {  // the lengths must fit the caches they index
      if (!fetch_ints(seq_lens, (size_t)B, lens, stream, &status)) return status;
      for (int b = 0; b < B; ++b)
        if (lens[b] < 0 || lens[b] > L_cap - N) return GLIDE_ERANGE;
    }
    if (!fetch_ints(parents, (size_t)B * N, par, stream, &status)) return status;
    if (!parents_ok(par, B, N)) return GLIDE_ERANGE;
  }
  a.target_argmax = target_argmax;
  a.cand = cand_tokens;
  a.parents = parents;
  a.seq_lens = seq_lens;
  a.seq_lens_out = seq_lens_out;
  a.accept_len = accept_len;
  a.last_node = last_node;
  a.bonus = bonus;
  a.path = path;
  a.B = B;
  a.N = N;
  a.H = H;
  a.L_cap = L_cap;
  a.layers = layers;
  a.row_bytes = D * (dtype == GLIDE_BF16 ? 2 : 4);
  return hip_status(glide::launch_verify_commit(logits, V, a, stream));
}

static int rows_matmul_impl(const void* a, const void* w, void* out, int M, int K, int N,
                            int out_dtype, bool packed, hipStream_t stream) {
  if (!a || !w || !out || !aligned16(a) || !aligned16(w)) return GLIDE_EINVAL;
  if (!rows_matmul_sizes_ok(M, K, N)) return GLIDE_EINVAL;
  if (out_dtype != GLIDE_BF16 && out_dtype != GLIDE_F32) return GLIDE_EINVAL;
  return hip_status(glide::launch_rows_matmul(a, w, out, M, K, N, out_dtype == GLIDE_BF16, packed, stream));
}

int glide_rows_matmul(const void* a, const void* w_t, void* out, int M, int K, int N, int out_dtype,
                      hipStream_t stream) {
  return rows_matmul_impl(a, w_t, out, M, K, N, out_dtype, false, stream);
}

size_t glide_rows_weights_packed_bytes(int K, int N) {
  return rows_matmul_sizes_ok(1, K, N) ? glide::packed_rows_weights_bytes(K, N) : 0;
}

int glide_pack_rows_weights(const void* w_t, void* w_packed, int K, int N, hipStream_t stream) {
  if (!w_t || !w_packed || !aligned16(w_t) || !aligned16(w_packed)) return GLIDE_EINVAL;
  if (!rows_matmul_sizes_ok(1, K, N)) return GLIDE_EINVAL;
  return hip_status(glide::launch_pack_rows_weights(w_t, w_packed, K, N, stream));
}

int glide_rows_matmul_packed(const void* a, const void* w_packed, void* out, int M, int K, int N,
                             int out_dtype, hipStream_t stream) {
  return rows_matmul_impl(a, w_packed, out, M, K, N, out_dtype, true, stream);
}

size_t glide_cross_block_workspace(int B, int Nq, int d_D, int H, int D, int L_cap) {
  CrossPlan p;
  return cross_block_plan(B, Nq, d_D, H, D, L_cap, &p) ? p.bytes : 0;
}

static int cross_block_impl(const void* hidden, const void* wq_t, const void* k_cache,
                            const void* v_cache, const int32_t* seq_lens, const void* wo_t, void* out,
                            int B, int Nq, int d_D, int H, int D, int L_cap, float scale,
                            void* workspace, size_t ws_bytes, bool packed, hipStream_t stream) {
  if (!hidden || !wq_t || !k_cache || !v_cache || !seq_lens || !wo_t || !out || !workspace)
    return GLIDE_EINVAL;
  if (!aligned16(hidden) || !aligned16(wq_t) || !aligned16(wo_t) || !aligned16(workspace))
    return GLIDE_EINVAL;
  if (!isfinite(scale)) return GLIDE_EINVAL;
  CrossPlan p;
  if (!cross_block_plan(B, Nq, d_D, H, D, L_cap, &p) || ws_bytes < p.bytes) return GLIDE_EINVAL;
  if (validate_enabled()) {
    int status = GLIDE_OK;
    std::vector<int32_t> lens;
    if (!fetch_ints(seq_lens, (size_t)B, lens, stream, &status)) return status;
    for (int b = 0; b < B; ++b)
      if (lens[b] < 0 || lens[b] > L_cap) return GLIDE_ERANGE;
  }
  char* ws = (char*)workspace;
  void* q = ws + p.q_off;
  void* heads = ws + p.heads_off;
  const int M = B * Nq;
  hipError_t e = glide::launch_rows_matmul(hidden, wq_t, q, M, d_D, H * D, true, packed, stream);
  if (e != hipSuccess) return hip_status(e);
  const glide::AttnArgs a = attn_args(q, k_cache, v_cache, seq_lens, nullptr, heads, B, Nq, H, D,
                                      L_cap, scale, p.attn, ws + p.attn_off);
  e = glide::launch_tree_attn(a, true, stream);
  if (e != hipSuccess) return hip_status(e);
  return hip_status(glide::launch_rows_matmul(heads, wo_t, out, M, H * D, d_D, true, packed, stream));
}

int glide_cross_block(const void* hidden, const void* wq_t, const void* k_cache, const void* v_cache,
                      const int32_t* seq_lens, const void* wo_t, void* out, int B, int Nq, int d_D,
                      int H, int D, int L_cap, float scale, void* workspace, size_t ws_bytes,
                      hipStream_t stream) {
  return cross_block_impl(hidden, wq_t, k_cache, v_cache, seq_lens, wo_t, out, B, Nq, d_D, H, D, L_cap,
                          scale, workspace, ws_bytes, false, stream);
}

int glide_cross_block_packed(const void* hidden, const void* wq_packed, const void* k_cache,
                             const void* v_cache, const int32_t* seq_lens, const void* wo_packed,
                             void* out, int B, int Nq, int d_D, int H, int D, int L_cap, float scale,
                             void* workspace, size_t ws_bytes, hipStream_t stream) {
  return cross_block_impl(hidden, wq_packed, k_cache, v_cache, seq_lens, wo_packed, out, B, Nq, d_D, H,
                          D, L_cap, scale, workspace, ws_bytes, true, stream);
}

int glide_block_attn(const void* q, const void* k_cache, const void* v_cache, void* out, int B, int T,
                     int H, int D, int L_cap, int block, float scale, hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !out) return GLIDE_EINVAL;
  if (B < 1 || B > 65535 || H < 1 || T < 1 || T > L_cap || D != glide::kHeadDim || block < 1)
    return GLIDE_EINVAL;
  if ((T + 63) / 64 > 65535 || L_cap > kMaxKeys || !isfinite(scale)) return GLIDE_EINVAL;
  if ((double)B * H * ((T + 63) / 64) > 2147483647.0) return GLIDE_EINVAL;  // linear workgroup ids
  if ((double)B * H * (double)L_cap * D > 9.0e18 || (double)B * T * H * D > 9.0e18) return GLIDE_EINVAL;
  glide::BlockAttnArgs a{};
  a.q = q;
  a.k = k_cache;
  a.v = v_cache;
  a.out = out;
  a.B = B;
  a.T = T;
  a.H = H;
  a.L_cap = L_cap;
  a.block = block;
  const double sc = scale > 0.f ? (double)scale : 1.0 / sqrt((double)D);
  a.scale_log2 = (float)(sc * 1.4426950408889634);  // log2(e)
  return hip_status(glide::launch_block_attn(a, stream));
}

int spec_sample_verify(const int32_t* draft_tokens, const float* draft_probs, const float* target_probs,
                       const float* uniforms, int B, int gamma, int V, int32_t* accept_len,
                       int32_t* next_token, hipStream_t stream) {
  if (!draft_tokens || !draft_probs || !target_probs || !uniforms || !accept_len || !next_token)
    return GLIDE_EINVAL;
  if (B < 1 || gamma < 1 || gamma > glide::kMaxSpecGamma || V < 1 || V > glide::kMaxSpecVocab)
    return GLIDE_EINVAL;
  if ((double)B * (gamma + 1) * V > 9.0e18) return GLIDE_EINVAL;
  return hip_status(glide::launch_spec_sample(draft_tokens, draft_probs, target_probs, uniforms, B, gamma,
                                              V, accept_len, next_token, stream));
}

double glide_expected_speedup(double alpha, int gamma, double c) {
  if (!(alpha >= 0.0 && alpha <= 1.0) || gamma < 1 || !(c >= 0.0)) return NAN;
  if (alpha == 1.0) return (gamma + 1) / (gamma * c + 1.0);
  return (1.0 - pow(alpha, gamma + 1)) / ((1.0 - alpha) * (gamma * c + 1.0));
}

}  // extern "C"
