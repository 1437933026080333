// Chain verification with speculative sampling (arXiv 2402.02082, Sec. 3:
// the accepted draft tokens plus one target token extend the prefix, and the
// emitted tokens follow the target's sampling distribution; Sec. 5.1: the
// GliDe-only experiments verify gamma = 5 chains this way).
//
// One 1024-thread workgroup per sequence.  Proposal token x_i is accepted when
// r_i * p_D(x_i) < p_T(x_i) (float32), tested for every position at once; the
// first rejection j picks the residual row max(0, p_T_j - p_D_j), no
// rejection picks the target row after the last token.  The token is drawn by
// inverse CDF over fixed-point weights floor(p * 2^32): integer sums do not
// depend on the order of summation, so the draw is a function of the inputs
// alone (each thread sums a contiguous chunk, a block-wide exclusive scan of
// the chunk sums locates the chunk that holds floor(u * W), and its thread
// walks it).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace glide {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ uint64_t fixed_weight(float p) {
  // p >= 0 (negatives count as 0); p * 2^32 is exact in float64
  return p > 0.f ? (uint64_t)((double)p * 4294967296.0) : 0;
}

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int d) {
  const uint32_t lo = __shfl_up((uint32_t)v, d), hi = __shfl_up((uint32_t)(v >> 32), d);
  return ((uint64_t)hi << 32) | lo;
}

// Weight of token v in the chosen row: the residual (mode 0) or the target
// row itself (mode 1).
__device__ __forceinline__ uint64_t row_weight(const float* pt, const float* pd, int v, int mode) {
  if (mode == 1) return fixed_weight(pt[v]);
  const float r = pt[v] - pd[v];
  return fixed_weight(r > 0.f ? r : 0.f);
}

// Exclusive block-wide scan of one uint64 per thread; also returns the total.
__device__ uint64_t block_exclusive_scan(uint64_t x, uint64_t* total) {
  __shared__ uint64_t wave_sum[kWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t incl = x;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t y = shfl_up_u64(incl, d);
    if (lane >= d) incl += y;
  }
  if (lane == 63) wave_sum[wave] = incl;
  __syncthreads();
  uint64_t before = 0, all = 0;
  for (int w = 0; w < kWaves; ++w) {
    const uint64_t s = wave_sum[w];
    if (w < wave) before += s;
    all += s;
  }
  __syncthreads();  // wave_sum is reused by the next call
  *total = all;
  return before + incl - x;
}

// Up to kHeld tokens per thread (V <= 4 * kThreads * 8 = 32768): the pass
// that sums a thread's chunk also parks the chosen row's per-token values in
// LDS (element-major, so a wave's stores are conflict-free), and the owner of
// the drawn chunk searches them there instead of reading the rows again.
constexpr int kHeld = 32;

__device__ uint64_t held_weight(float* held, const float* pt, const float* pd, int v0, int v1, int mode,
                                bool vec) {
  const int tid = threadIdx.x;
  uint64_t sum = 0;
  if (vec) {
#pragma unroll 2
    for (int i = 0; i < kHeld; i += 4) {
      const int v = v0 + i;
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f), d = a;
      if (v < v1) {
        a = *(const float4*)(pt + v);
        if (mode == 0) d = *(const float4*)(pd + v);
      }
      const float av[4] = {a.x, a.y, a.z, a.w}, dv[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float p = av[e];
        if (mode == 0) {
          const float r = av[e] - dv[e];
          p = r > 0.f ? r : 0.f;
        }
        held[(i + e) * kThreads + tid] = p;
        sum += fixed_weight(p);
      }
    }
  } else {
    for (int i = 0; i < kHeld; ++i) {
      const int v = v0 + i;
      float p = 0.f;
      if (v < v1) {
        p = pt[v];
        if (mode == 0) {
          const float r = p - pd[v];
          p = r > 0.f ? r : 0.f;
        }
      }
      held[i * kThreads + tid] = p;
      sum += fixed_weight(p);
    }
  }
  return sum;
}

__device__ int held_find(const float* held, int v0, int v1, uint64_t run, uint64_t t) {
  const int tid = threadIdx.x;
  int found = v1 - 1;
  bool done = false;
  for (int i = 0; i < kHeld && v0 + i < v1; ++i) {
    run += fixed_weight(held[i * kThreads + tid]);
    if (!done && run > t) {
      found = v0 + i;
      done = true;
    }
  }
  return found;
}

// Sum of the weights of tokens [v0, v1).
__device__ uint64_t chunk_weight(const float* pt, const float* pd, int v0, int v1, int mode, bool vec) {
  uint64_t sum = 0;
  if (vec) {
#pragma unroll 8
    for (int v = v0; v < v1; v += 4) {
      const float4 a = *(const float4*)(pt + v);
      const float4 d = mode == 1 ? a : *(const float4*)(pd + v);
      if (mode == 1) {
        sum += fixed_weight(a.x) + fixed_weight(a.y) + fixed_weight(a.z) + fixed_weight(a.w);
      } else {
        const float r0 = a.x - d.x, r1 = a.y - d.y, r2 = a.z - d.z, r3 = a.w - d.w;
        sum += fixed_weight(r0 > 0.f ? r0 : 0.f) + fixed_weight(r1 > 0.f ? r1 : 0.f) +
               fixed_weight(r2 > 0.f ? r2 : 0.f) + fixed_weight(r3 > 0.f ? r3 : 0.f);
      }
    }
  } else {
    for (int v = v0; v < v1; ++v) sum += row_weight(pt, pd, v, mode);
  }
  return sum;
}

// The first token of [v0, v1) whose running weight (from `run`) exceeds t;
// the running sum is taken without an early exit so the loads go out
// together.
__device__ int chunk_find(const float* pt, const float* pd, int v0, int v1, int mode, bool vec,
                          uint64_t run, uint64_t t) {
  int found = v1 - 1;
  bool done = false;
  if (vec) {
#pragma unroll 8
    for (int v = v0; v < v1; v += 4) {
      const float4 a = *(const float4*)(pt + v);
      const float4 d = mode == 1 ? a : *(const float4*)(pd + v);
      const float av[4] = {a.x, a.y, a.z, a.w}, dv[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float p = av[e];
        if (mode == 0) {
          const float r = av[e] - dv[e];
          p = r > 0.f ? r : 0.f;
        }
        run += fixed_weight(p);
        if (!done && run > t) {
          found = v + e;
          done = true;
        }
      }
    }
  } else {
    for (int v = v0; v < v1; ++v) {
      run += row_weight(pt, pd, v, mode);
      if (!done && run > t) {
        found = v;
        done = true;
      }
    }
  }
  return found;
}

template <bool KEEP>
__global__ __launch_bounds__(kThreads) void spec_sample_kernel(const int32_t* __restrict__ draft_tokens,
                                                               const float* __restrict__ p_draft,
                                                               const float* __restrict__ p_target,
                                                               const float* __restrict__ uniforms,
                                                               int gamma, int V,
                                                               int32_t* __restrict__ accept_len,
                                                               int32_t* __restrict__ next_token) {
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const float* u = uniforms + (size_t)b * (gamma + 1);
  __shared__ int first_reject;

  // Acceptance tests of every position (gamma <= 64: wave 0).
  if (tid < 64) {
    bool rejected = false;
    if (lane < gamma) {
      int x = draft_tokens[(size_t)b * gamma + lane];
      x = x < 0 ? 0 : (x >= V ? V - 1 : x);
      const float pd = p_draft[((size_t)b * gamma + lane) * V + x];
      const float pt = p_target[((size_t)b * (gamma + 1) + lane) * V + x];
      rejected = !(u[lane] * pd < pt);
    }
    const uint64_t rej = __ballot(rejected);
    if (lane == 0) first_reject = rej ? __ffsll((long long)rej) - 1 : gamma;
  }
  __syncthreads();
  const int j = first_reject;
  const float* pt = p_target + ((size_t)b * (gamma + 1) + j) * V;
  const float* pd = p_draft + ((size_t)b * gamma + (j < gamma ? j : 0)) * V;

  // Contiguous chunks of a multiple of 4 tokens per thread; with V % 4 == 0
  // and 16-byte aligned arrays every chunk is read with float4 loads.
  const int chunk = ((V + 4 * kThreads - 1) / (4 * kThreads)) * 4;
  const int v0 = min(V, tid * chunk), v1 = min(V, v0 + chunk);
  const bool vec = (V & 3) == 0 && ((((uintptr_t)p_target) | ((uintptr_t)p_draft)) & 15) == 0;
  int mode = j < gamma ? 0 : 1;
  // KEEP (chunk <= kHeld): the chunk fits the LDS copy, so the rows are read once
  __shared__ float held[KEEP ? kHeld * kThreads : 1];
  uint64_t total = 0, mine = 0, before = 0;
  for (int pass = 0; pass < 2; ++pass) {
    mine = KEEP ? held_weight(held, pt, pd, v0, v1, mode, vec) : chunk_weight(pt, pd, v0, v1, mode, vec);
    before = block_exclusive_scan(mine, &total);
    if (total > 0 || mode == 1) break;
    mode = 1;  // a residual of zero weight: draw from the target row itself
  }
  if (total == 0) {
    if (tid == 0) {
      accept_len[b] = j;
      next_token[b] = 0;
    }
    return;
  }
  uint64_t t = (uint64_t)((double)u[gamma] * (double)total);
  if (t >= total) t = total - 1;
  if (before <= t && t < before + mine) {
    accept_len[b] = j;
    // the owner reads back its own LDS entries (no barrier needed)
    next_token[b] = KEEP ? held_find(held, v0, v1, before, t) : chunk_find(pt, pd, v0, v1, mode, vec, before, t);
  }
}

}  // namespace

hipError_t launch_spec_sample(const int32_t* draft_tokens, const float* p_draft, const float* p_target,
                              const float* uniforms, int B, int gamma, int V, int32_t* accept_len,
                              int32_t* next_token, hipStream_t stream) {
  const int chunk = ((V + 4 * kThreads - 1) / (4 * kThreads)) * 4;
  if (chunk <= kHeld)
    hipLaunchKernelGGL(spec_sample_kernel<true>, dim3(B), dim3(kThreads), 0, stream, draft_tokens, p_draft,
                       p_target, uniforms, gamma, V, accept_len, next_token);
  else
    hipLaunchKernelGGL(spec_sample_kernel<false>, dim3(B), dim3(kThreads), 0, stream, draft_tokens, p_draft,
                       p_target, uniforms, gamma, V, accept_len, next_token);
  return hipGetLastError();
}

}  // namespace glide
