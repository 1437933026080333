// Verify commit (arXiv 2402.02082): greedy acceptance of the candidate tree
// followed by the KV cache commit.  Sec. 3: the first accepted proposal
// tokens plus one token of the target's own extend the prefix; Sec. 4.1:
// after a verification step only the accepted tokens' cache rows are kept;
// Sec. 4.2: a tree candidate is accepted when its whole root path is.
//
// One wave per (sequence, layer, head).  Every wave first works out its
// sequence's acceptance (one lane per node, ancestor masks by pointer
// doubling -- a few dozen instructions, cheaper than a second launch), then
// moves the accepted path's K and V rows of its (layer, head) slab to the
// rows right behind the prefix.  The path's node at depth d + 1 sits at row
// L + n_{d+1} >= L + d, so a destination row is never the source of a deeper
// slot; all sources of a batch are loaded before its stores, so a
// destination that is the source of a shallower slot is read first.  Each
// slab is moved by exactly one wave.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace glide {
namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

constexpr int kWaves = 4;
constexpr int kIter = 16;  // 16-byte loads per matrix and lane in one batch

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl((uint32_t)v, src), hi = __shfl((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)(v >> 32), m);
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    v = o > v ? o : v;
  }
  return v;
}

__global__ __launch_bounds__(64 * kWaves) void verify_commit_kernel(CommitArgs args) {
  const int b = blockIdx.z, layer = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = blockIdx.x * kWaves + wave;
  const int N = args.N;
  const int32_t* ta = args.target_argmax + (size_t)b * (N + 1);

  // Acceptance: node n is accepted iff every node on its root path matches.
  int p = -1;
  bool match = false;
  uint64_t anc = 0;
  if (lane < N) {
    p = args.parents[(size_t)b * N + lane];
    if (p < -1 || p >= lane) p = -1;
    match = args.cand[(size_t)b * N + lane] == ta[p + 1];
    anc = 1ull << lane;
  }
  const uint64_t matched = __ballot(match);
#pragma unroll
  for (int round = 0; round < 6; ++round) {
    const int src = p < 0 ? lane : p;
    const uint64_t a_up = shfl_u64(anc, src);
    const int p_up = __shfl(p, src);
    if (p >= 0) {
      anc |= a_up;
      p = p_up;
    }
  }
  const bool accepted = lane < N && (anc & ~matched) == 0;
  const int depth = __popcll(anc);
  const uint64_t key = wave_max_u64(accepted ? (((uint64_t)depth << 8) | (uint64_t)(255 - lane)) : 0);
  const int a = (int)(key >> 8);
  const int last = key ? 255 - (int)(key & 255) : -1;
  const uint64_t path_mask = last >= 0 ? shfl_u64(anc, last) : 0;
  // slot (depth - 1) of every path node, and the node in every slot
  const bool on_path = (path_mask >> lane) & 1;
  const int rank = __popcll(path_mask & ((1ull << lane) - 1));
  __shared__ int node_of[kWaves][64];
  if (on_path) node_of[wave][rank] = lane;

  if (blockIdx.x == 0 && layer == 0 && wave == 0) {
    if (lane == 0) {
      args.accept_len[b] = a;
      args.seq_lens_out[b] = args.seq_lens[b] + a;
      if (args.last_node) args.last_node[b] = last;
      if (args.bonus) args.bonus[b] = ta[last + 1];
    }
    if (args.path) {
      if (on_path) args.path[(size_t)b * N + rank] = lane;
      if (lane >= a && lane < N) args.path[(size_t)b * N + lane] = -1;
    }
  }
  __syncthreads();
  if (layer >= args.layers || h >= args.H || a == 0) return;

  const int R = args.row_bytes;                 // 256 (bf16) or 512 (fp32)
  const int lanes_per_row = R / 16;
  const int rows_per_load = 64 / lanes_per_row;
  const int chunk = lane % lanes_per_row, q = lane / lanes_per_row;
  const int L = min(max(args.seq_lens[b], 0), args.L_cap - N);
  const size_t slab = (((size_t)b * args.H + h) * args.L_cap + L) * R + chunk * 16;
  char* kb = args.k[layer] + slab;
  char* vb = args.v[layer] + slab;

  for (int s0 = 0; s0 < a; s0 += kIter * rows_per_load) {
    u32x4_t kx[kIter], vx[kIter];
#pragma unroll
    for (int i = 0; i < kIter; ++i) {
      const int d = s0 + i * rows_per_load + q;
      const int n = d < a ? node_of[wave][d] : d;
      if (n != d) {  // a path that starts down the chain keeps those rows in place
        kx[i] = *(const u32x4_t*)(kb + (size_t)n * R);
        vx[i] = *(const u32x4_t*)(vb + (size_t)n * R);
      }
    }
#pragma unroll
    for (int i = 0; i < kIter; ++i) {
      const int d = s0 + i * rows_per_load + q;
      const int n = d < a ? node_of[wave][d] : d;
      if (n != d) {
        *(u32x4_t*)(kb + (size_t)d * R) = kx[i];
        *(u32x4_t*)(vb + (size_t)d * R) = vx[i];
      }
    }
  }
}

}  // namespace

hipError_t launch_verify_commit(const float* logits, int V, const CommitArgs& a, hipStream_t stream) {
  hipError_t e = launch_argmax_rows(logits, a.B * (a.N + 1), V, a.target_argmax, stream);
  if (e != hipSuccess) return e;
  const dim3 grid((a.H + kWaves - 1) / kWaves, a.layers > 0 ? a.layers : 1, a.B);
  hipLaunchKernelGGL(verify_commit_kernel, grid, dim3(64 * kWaves), 0, stream, a);
  return hipGetLastError();
}

}  // namespace glide
