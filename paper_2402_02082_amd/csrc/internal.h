// Internal launch interface between the C ABI (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace glide {

constexpr int kHeadDim = 128;
constexpr int kMaxNodes = 64;
constexpr int kMaxSplits = 64;
constexpr int kNumCU = 256;        // MI355X compute units (split heuristic)
constexpr int kChunkQuantum = 32;  // split boundaries are multiples of this
constexpr int kMinChunk = 128;     // smallest split the automatic plan makes

// How the keys of one (sequence, head) are divided between workgroups.
struct AttnPlan {
  int splits;       // workgroups per (sequence, head)
  int chunk;        // keys per workgroup (multiple of kChunkQuantum)
  size_t ws_bytes;  // workspace for the partial states (0 if splits == 1)
  size_t part_o_off, part_ml_off;
};

AttnPlan plan_tree_attn(int B, int N, int H, int L_cap, int max_splits);

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* seq_lens;
  const int32_t* parents;  // nullptr: cross mode
  void* out;
  float* part_o;           // [B, H, splits, N, D]
  float2* part_ml;         // [B, H, splits, N] (running max in log2 units, sum)
  int B, N, H, L_cap, chunk, splits;
  float scale_log2;        // softmax scale * log2(e)
};

hipError_t launch_tree_attn(const AttnArgs& a, bool bf16, hipStream_t stream);

size_t cape_workspace_bytes(int B, int gamma, int V);
hipError_t launch_cape_expand(const float* probs, int B, int gamma, int V, int k,
                              int fixed, int n_max, int32_t* tokens,
                              int32_t* parents, int32_t* n_nodes, void* ws,
                              hipStream_t stream);

hipError_t launch_argmax_rows(const float* logits, int rows, int V, int32_t* idx,
                              hipStream_t stream);

// out[m, n] = sum_k a[m, k] w_t[n, k] (bf16 in, fp32 accumulation); up to
// kMaxMatmulRows rows per launch, more rows loop.
constexpr int kMaxMatmulRows = 64;
constexpr int kMaxMatmulK = 1 << 20;
hipError_t launch_rows_matmul(const void* a, const void* w_t, void* out, int M, int K, int N,
                              bool out_bf16, hipStream_t stream);

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
