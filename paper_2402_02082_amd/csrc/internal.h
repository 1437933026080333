// Internal launch interface between the C ABI (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "attn.h"

namespace glide {

size_t cape_workspace_bytes(int B, int gamma, int V);
hipError_t launch_cape_expand(const float* probs, int B, int gamma, int V, int k,
                              int fixed, int n_max, int32_t* tokens,
                              int32_t* parents, int32_t* n_nodes, void* ws,
                              hipStream_t stream);

hipError_t launch_argmax_rows(const float* logits, int rows, int V, int32_t* idx,
                              hipStream_t stream);

// out[m, n] = sum_k a[m, k] w_t[n, k] (bf16 in, fp32 accumulation); up to
// kMaxMatmulRows rows per launch, more rows loop.
constexpr int kMaxMatmulRows = 128;
constexpr int kMaxMatmulK = 1 << 20;
hipError_t launch_rows_matmul(const void* a, const void* w, void* out, int M, int K, int N,
                              bool out_bf16, bool packed, hipStream_t stream);
// Bytes of the packed copy of a [N, K] weight matrix: one 1 KB operand block
// per (16-row tile, 32-wide K step).
size_t packed_rows_weights_bytes(int K, int N);
hipError_t launch_pack_rows_weights(const void* w_t, void* packed, int K, int N, hipStream_t stream);

hipError_t launch_spec_sample(const int32_t* draft_tokens, const float* p_draft, const float* p_target,
                              const float* uniforms, int B, int gamma, int V, int32_t* accept_len,
                              int32_t* next_token, hipStream_t stream);
constexpr int kMaxSpecGamma = 64;
constexpr int kMaxSpecVocab = 1 << 20;

// Greedy acceptance plus the cache commit of every layer's K and V.
constexpr int kMaxLayers = 128;
struct CommitArgs {
  int32_t* target_argmax;  // [B, N + 1], written by the argmax launch
  const int32_t* cand;
  const int32_t* parents;
  const int32_t* seq_lens;
  int32_t* seq_lens_out;
  int32_t* accept_len;
  int32_t* last_node;      // nullable
  int32_t* bonus;          // nullable
  int32_t* path;           // nullable, [B, N]
  int B, N, H, L_cap, layers, row_bytes;
  char* k[kMaxLayers];
  char* v[kMaxLayers];
};

hipError_t launch_verify_commit(const float* logits, int V, const CommitArgs& a, hipStream_t stream);

hipError_t launch_tree_verify(const int32_t* target_argmax, const int32_t* cand,
                              const int32_t* parents, int B, int N,
                              int32_t* accept_len, int32_t* last_node,
                              int32_t* bonus, hipStream_t stream);

}  // namespace glide
