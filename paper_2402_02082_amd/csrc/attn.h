// Interface of the attention kernels (tree_attn.hip) to the C ABI.
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

// Arrival counters of the in-kernel split merge: one per (sequence, head),
// 128 bytes apart (counters sharing a cache line serialise their atomics),
// in a fixed block at offset 0 of every split workspace, so a buffer that
// serves calls of different shapes never finds partial states where a later
// call keeps counters.  The block must be zero before a workspace's first
// use; every call leaves it zero.  Only single-sequence calls merge this
// way (at most kCounterSlots heads); the others merge in a second launch.
constexpr int kCounterSlots = 2048;
constexpr int kCounterStride = 32;  // uint32 words: 128 bytes
constexpr size_t kCounterBytes = (size_t)kCounterSlots * kCounterStride * 4;
// Words 1..8 of a head's counter slot flag the (split, wave) pieces whose
// states did not fit fp16 (bit 4 * split + wave; up to 64 splits).
constexpr int kWideFlagWords = 8;

// How the keys of one (sequence, head) are divided between workgroups.
struct AttnPlan {
  int splits;       // workgroups per (sequence, head)
  int chunk;        // keys per workgroup (multiple of kChunkQuantum)
  size_t ws_bytes;  // workspace: counters + partial states (0 if splits == 1)
  size_t counters_off, part_o_off, part_ml_off, part_h_off;
  bool merge_in_kernel;  // the last split to finish merges (else a second launch)
  bool half_states;      // bf16 states exchanged as fp16 o / L (in-kernel merge, N >= 8)
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
  uint16_t* part_h;        // [B, H, splits, N, D] fp16 (in-kernel merge of bf16 calls)
  unsigned* counters;      // arrival counters (in-kernel merge), else nullptr
  int B, N, H, L_cap, chunk, splits;
  float scale_log2;        // softmax scale * log2(e)
};

hipError_t launch_tree_attn(const AttnArgs& a, bool bf16, hipStream_t stream);

// Block-masked cross attention of draft training: query position p attends
// to key positions [0, block * floor(p / block)).
struct BlockAttnArgs {
  const void* q;    // [B, T, H, D] bf16
  const void* k;    // [B, H, L_cap, D] bf16
  const void* v;
  void* out;        // [B, T, H, D] bf16
  int B, T, H, L_cap, block;
  float scale_log2;
};

hipError_t launch_block_attn(const BlockAttnArgs& a, hipStream_t stream);

}  // namespace glide
