// CaPE proposal expansion on the GPU (arXiv 2402.02082, Sec. 4.2,
// "Proposal Expansion"; linearisation from "Verification of Expanded
// Proposals"; verification budget from Sec. 5.3; fixed-size variant from
// Sec. 5.4).
//
// Two kernels:
//   cape_top8      one workgroup per draft row: the 8 best (prob desc, id asc)
//                  tokens of the row -- the proposal token and the largest
//                  possible expansion set (S(p) <= 7).
//   cape_assemble  one wave per sequence: S(p) sizes, budget cut, and the
//                  linearised parent-indexed tree.
// Every decision is an exact comparison of the float32 inputs (keys are the
// order-preserving integer image of the float, ties broken by token id), so
// the result is bit-exact by construction.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace glide {
namespace {

constexpr int kTopK = 8;
constexpr int kThreads = 256;

// Order-preserving map float32 -> uint32 (+0 and -0 map to the same value).
__device__ __forceinline__ uint32_t ordered_bits(float x) {
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float from_ordered_bits(uint32_t o) {
  const uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  return __uint_as_float(u);
}

// Larger key = more probable token; equal probabilities: lower id is larger.
__device__ __forceinline__ uint64_t rank_key(float p, int id) {
  return ((uint64_t)ordered_bits(p) << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)id);
}

__device__ __forceinline__ int key_id(uint64_t key) {
  return (int)(0xFFFFFFFFu - (uint32_t)key);
}

// Insert into a descending list of kTopK keys held in registers.
__device__ __forceinline__ void insert_key(uint64_t (&top)[kTopK], uint64_t key) {
  if (key <= top[kTopK - 1]) return;
  top[kTopK - 1] = key;
#pragma unroll
  for (int j = kTopK - 1; j > 0; --j) {
    const uint64_t hi = top[j - 1], lo = top[j];
    const bool sw = lo > hi;
    top[j - 1] = sw ? lo : hi;
    top[j] = sw ? hi : lo;
  }
}

__global__ __launch_bounds__(kThreads) void cape_top8(const float* __restrict__ probs, int V,
                                                      uint64_t* __restrict__ top_out) {
  const int row = blockIdx.x, tid = threadIdx.x;
  const float* p = probs + (size_t)row * V;
  uint64_t top[kTopK];
#pragma unroll
  for (int j = 0; j < kTopK; ++j) top[j] = 0;  // below every real key

  if ((V & 3) == 0 && (((uintptr_t)p) & 15) == 0) {
    const float4* p4 = (const float4*)p;
    for (int i = tid; i < V / 4; i += kThreads) {
      const float4 x = p4[i];
      insert_key(top, rank_key(x.x, 4 * i));
      insert_key(top, rank_key(x.y, 4 * i + 1));
      insert_key(top, rank_key(x.z, 4 * i + 2));
      insert_key(top, rank_key(x.w, 4 * i + 3));
    }
  } else {
    for (int i = tid; i < V; i += kThreads) insert_key(top, rank_key(p[i], i));
  }

  // Tree merge of the 256 per-thread lists through LDS.
  __shared__ uint64_t lists[kThreads][kTopK];
#pragma unroll
  for (int j = 0; j < kTopK; ++j) lists[tid][j] = top[j];
  __syncthreads();
  for (int stride = kThreads / 2; stride > 0; stride >>= 1) {
    if (tid < stride) {
#pragma unroll
      for (int j = 0; j < kTopK; ++j) insert_key(top, lists[tid + stride][j]);
    }
    __syncthreads();
    if (tid < stride) {
#pragma unroll
      for (int j = 0; j < kTopK; ++j) lists[tid][j] = top[j];
    }
    __syncthreads();
  }
  if (tid < kTopK) top_out[(size_t)row * kTopK + tid] = lists[0][tid];
}

// S(p): 7, 5, 3, 1 on (0, 0.3], (0.3, 0.6], (0.6, 0.8], (0.8, 1].
__device__ __forceinline__ int expansion_size(float p) {
  if (p <= 0.3f) return 7;
  if (p <= 0.6f) return 5;
  if (p <= 0.8f) return 3;
  return 1;
}

// One wave per sequence.  Candidate c enumerates (position i, rank r) in
// linearisation order; its confidence key is the top-8 key itself.
__global__ __launch_bounds__(64) void cape_assemble(const uint64_t* __restrict__ top, int gamma, int V,
                                                    int k, int fixed, int n_max,
                                                    int32_t* __restrict__ tokens,
                                                    int32_t* __restrict__ parents,
                                                    int32_t* __restrict__ n_nodes) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const uint64_t* tb = top + (size_t)b * gamma * kTopK;

  __shared__ int sizes[kMaxNodes];
  __shared__ int base[kMaxNodes + 1];
  __shared__ uint64_t cand_key[kMaxNodes * 7];
  __shared__ int cand_pos[kMaxNodes * 7];

  if (lane < gamma) {
    const uint64_t k0 = tb[lane * kTopK];
    int K;
    if (fixed) {
      K = k;
    } else {
      K = expansion_size(from_ordered_bits((uint32_t)(k0 >> 32)));
      if (k > 0) K = min(K, k);
    }
    sizes[lane] = min(K, V - 1);
    tokens[(size_t)b * n_max + lane] = key_id(k0);
    parents[(size_t)b * n_max + lane] = lane - 1;
  }
  __syncthreads();
  if (lane == 0) {
    int acc = 0;
    for (int i = 0; i < gamma; ++i) {
      base[i] = acc;
      acc += sizes[i];
    }
    base[gamma] = acc;
  }
  __syncthreads();
  const int C = base[gamma];
  for (int cidx = lane; cidx < C; cidx += 64) {
    int i = 0;
    while (base[i + 1] <= cidx) ++i;
    const int r = cidx - base[i] + 1;
    cand_key[cidx] = tb[i * kTopK + r];
    cand_pos[cidx] = i;
  }
  __syncthreads();

  const int budget = n_max - gamma;
  int written = 0;  // kept candidates in earlier chunks
  for (int cb = 0; cb < C; cb += 64) {
    const int cidx = cb + lane;
    bool kept = false;
    if (cidx < C) {
      if (C <= budget) {
        kept = true;
      } else {
        // Rank in (prob desc, position asc, rank asc): probability is the
        // high half of the key; cidx order is (position, rank) order.
        const uint32_t pc = (uint32_t)(cand_key[cidx] >> 32);
        int ahead = 0;
        for (int o = 0; o < C; ++o) {
          const uint32_t po = (uint32_t)(cand_key[o] >> 32);
          ahead += (po > pc) || (po == pc && o < cidx);
        }
        kept = ahead < budget;
      }
    }
    const uint64_t mask = __ballot(kept);
    if (kept) {
      const int slot = gamma + written + __popcll(mask & ((1ull << lane) - 1ull));
      tokens[(size_t)b * n_max + slot] = key_id(cand_key[cidx]);
      parents[(size_t)b * n_max + slot] = cand_pos[cidx] - 1;
    }
    written += __popcll(mask);
  }
  const int n = gamma + written;
  for (int j = n + lane; j < n_max; j += 64) {
    tokens[(size_t)b * n_max + j] = -1;
    parents[(size_t)b * n_max + j] = -1;
  }
  if (lane == 0) n_nodes[b] = n;
}

}  // namespace

size_t cape_workspace_bytes(int B, int gamma) {
  return (size_t)B * gamma * kTopK * sizeof(uint64_t);
}

hipError_t launch_cape_expand(const float* probs, int B, int gamma, int V, int k, int fixed,
                              int n_max, int32_t* tokens, int32_t* parents, int32_t* n_nodes,
                              void* ws, hipStream_t stream) {
  uint64_t* top = (uint64_t*)ws;
  hipLaunchKernelGGL(cape_top8, dim3(B * gamma), dim3(kThreads), 0, stream, probs, V, top);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cape_assemble, dim3(B), dim3(64), 0, stream, top, gamma, V, k, fixed, n_max,
                     tokens, parents, n_nodes);
  return hipGetLastError();
}

}  // namespace glide
