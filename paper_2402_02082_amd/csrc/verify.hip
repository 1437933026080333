// Greedy verification of a candidate tree (arXiv 2402.02082, Sec. 3: with
// greedy "speculative decoding" acceptance a proposed token is kept exactly
// when it equals the target's greedy token; Sec. 4.2 verifies the whole
// expanded proposal in one pass; Sec. 5.1 uses greedy acceptance for CaPE).
//
//   argmax_rows   one workgroup per logits row: the first index of the row
//                 maximum (a max over (order-preserving value, ~index)
//                 keys); 1024 threads while every row's workgroup fits on
//                 the chip at once (a 32000-entry row is one round of
//                 loads), 256 beyond that, so that no rows wait for a
//                 second round of workgroups.
//   tree_verify   one wave per sequence, one lane per node: a node is
//                 accepted iff every node on its root path matches, i.e. its
//                 ancestor-or-self bitmask has no non-matching bit; the
//                 deepest accepted node (lowest index on ties) wins.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace glide {
namespace {

__device__ __forceinline__ uint32_t ordered_bits(float x) {
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ uint64_t argmax_key(float x, int idx) {
  return ((uint64_t)ordered_bits(x) << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)idx);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl((uint32_t)v, src), hi = __shfl((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m > 0; m >>= 1) {
    const uint64_t o = shfl_xor_u64(v, m);
    v = o > v ? o : v;
  }
  return v;
}

// One workgroup of kThreads per row; each thread requests 8 float4 (32
// values) at once, so with 1024 threads a 32000-entry row is a single round
// of loads.
constexpr int kArgmaxVec = 8;

template <int kArgmaxThreads>
__global__ __launch_bounds__(kArgmaxThreads) void argmax_rows_kernel(const float* __restrict__ logits,
                                                                     int V, int32_t* __restrict__ idx) {
  const int row = blockIdx.x, tid = threadIdx.x;
  const float* p = logits + (size_t)row * V;
  uint64_t best = 0;
  if ((V & 3) == 0 && (((uintptr_t)p) & 15) == 0) {
    const float4* p4 = (const float4*)p;
    const int n4 = V / 4;
    for (int i0 = 0; i0 < n4; i0 += kArgmaxThreads * kArgmaxVec) {
      float4 x[kArgmaxVec];
#pragma unroll
      for (int u = 0; u < kArgmaxVec; ++u) {
        const int i = i0 + tid + kArgmaxThreads * u;
        x[u] = i < n4 ? p4[i] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < kArgmaxVec; ++u) {
        const int i = i0 + tid + kArgmaxThreads * u;
        if (i < n4) {
          uint64_t k0 = argmax_key(x[u].x, 4 * i), k1 = argmax_key(x[u].y, 4 * i + 1);
          uint64_t k2 = argmax_key(x[u].z, 4 * i + 2), k3 = argmax_key(x[u].w, 4 * i + 3);
          k0 = k1 > k0 ? k1 : k0;
          k2 = k3 > k2 ? k3 : k2;
          k0 = k2 > k0 ? k2 : k0;
          best = k0 > best ? k0 : best;
        }
      }
    }
  } else {
    for (int i = tid; i < V; i += kArgmaxThreads) {
      const uint64_t k = argmax_key(p[i], i);
      best = k > best ? k : best;
    }
  }
  best = wave_max_u64(best);
  __shared__ uint64_t per_wave[kArgmaxThreads / 64];
  if ((tid & 63) == 0) per_wave[tid >> 6] = best;
  __syncthreads();
  if (tid < 64) {
    uint64_t m = tid < kArgmaxThreads / 64 ? per_wave[tid] : 0;
    m = wave_max_u64(m);
    if (tid == 0) idx[row] = (int32_t)(0xFFFFFFFFu - (uint32_t)m);
  }
}

__global__ __launch_bounds__(64) void tree_verify_kernel(const int32_t* __restrict__ target_argmax,
                                                         const int32_t* __restrict__ cand,
                                                         const int32_t* __restrict__ parents, int N,
                                                         int32_t* __restrict__ accept_len,
                                                         int32_t* __restrict__ last_node,
                                                         int32_t* __restrict__ bonus) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const int32_t* ta = target_argmax + (size_t)b * (N + 1);
  int p = -1;
  bool match = false;
  uint64_t anc = 0;
  if (lane < N) {
    p = parents[(size_t)b * N + lane];
    if (p < -1 || p >= lane) p = -1;
    match = cand[(size_t)b * N + lane] == ta[p + 1];
    anc = 1ull << lane;
  }
  const uint64_t matched = __ballot(match);
  // Ancestor-or-self masks by pointer doubling (six rounds cover depth 64).
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
  // Deepest accepted node, then the lowest index.
  uint64_t key = accepted ? (((uint64_t)depth << 8) | (uint64_t)(255 - lane)) : 0;
  key = wave_max_u64(key);
  if (lane == 0) {
    const int len = (int)(key >> 8);
    const int last = key ? 255 - (int)(key & 255) : -1;
    accept_len[b] = len;
    if (last_node) last_node[b] = last;
    if (bonus) bonus[b] = ta[last + 1];
  }
}

}  // namespace

hipError_t launch_argmax_rows(const float* logits, int rows, int V, int32_t* idx,
                              hipStream_t stream) {
  // two 1024-thread workgroups fit on a CU
  if (rows <= 2 * kNumCU)
    hipLaunchKernelGGL(argmax_rows_kernel<1024>, dim3(rows), dim3(1024), 0, stream, logits, V, idx);
  else
    hipLaunchKernelGGL(argmax_rows_kernel<256>, dim3(rows), dim3(256), 0, stream, logits, V, idx);
  return hipGetLastError();
}

hipError_t launch_tree_verify(const int32_t* target_argmax, const int32_t* cand,
                              const int32_t* parents, int B, int N, int32_t* accept_len,
                              int32_t* last_node, int32_t* bonus, hipStream_t stream) {
  hipLaunchKernelGGL(tree_verify_kernel, dim3(B), dim3(64), 0, stream, target_argmax, cand, parents,
                     N, accept_len, last_node, bonus);
  return hipGetLastError();
}

}  // namespace glide
