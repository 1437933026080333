// CaPE proposal expansion on the GPU (arXiv 2402.02082, Sec. 4.2,
// "Proposal Expansion"; linearisation from "Verification of Expanded
// Proposals"; verification budget from Sec. 5.3; fixed-size variant from
// Sec. 5.4).
//
// Two kernels:
//   cape_top8_part  one workgroup per 4096-token part of a draft row: the 8
//                   best (prob desc, id asc) tokens of the part;
//   cape_assemble   one workgroup per sequence: merges the parts into the
//                   row's top 8 -- the proposal token and the largest possible
//                   expansion set (S(p) <= 7) -- then applies S(p), the budget
//                   cut and the linearisation into a parent-indexed tree.
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

// Top 8 of two descending lists of 8, descending (bitonic merge: the
// element-wise max of a and reversed b holds the 8 largest keys as a bitonic
// sequence, which three compare-exchange stages sort).
__device__ __forceinline__ void merge_top8(uint64_t (&a)[kTopK], const uint64_t (&b)[kTopK]) {
#pragma unroll
  for (int i = 0; i < kTopK; ++i) a[i] = a[i] > b[kTopK - 1 - i] ? a[i] : b[kTopK - 1 - i];
#pragma unroll
  for (int dist = kTopK / 2; dist > 0; dist >>= 1)
#pragma unroll
    for (int i = 0; i < kTopK; ++i)
      if ((i & dist) == 0) {
        const uint64_t x = a[i], y = a[i + dist];
        a[i] = x > y ? x : y;
        a[i + dist] = x > y ? y : x;
      }
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

// Butterfly merge of the lists held by the lanes [0, width) of a wave; every
// lane ends with the top 8 of its aligned group of `width` lanes.
__device__ __forceinline__ void wave_merge_top8(uint64_t (&top)[kTopK], int width) {
  for (int m = 1; m < width; m <<= 1) {
    uint64_t other[kTopK];
#pragma unroll
    for (int j = 0; j < kTopK; ++j) other[j] = shfl_xor_u64(top[j], m);
    merge_top8(top, other);
  }
}

// Elements of a draft row handled by one workgroup: 256 threads x 16.
constexpr int kPart = kThreads * 16;

__device__ __forceinline__ int parts_per_row(int V) { return (V + kPart - 1) / kPart; }

// Top-8 keys of one 4096-element part of one draft row.  Every thread
// requests its 16 elements at once and keeps its own top 8; the lists are
// merged with bitonic top-8 merges, across lanes by shuffles and across the
// four waves through LDS.
__global__ __launch_bounds__(kThreads) void cape_top8_part(const float* __restrict__ probs, int V,
                                                           uint64_t* __restrict__ top_out) {
  const int part = blockIdx.x, row = blockIdx.y, tid = threadIdx.x;
  const int P = gridDim.x;
  const float* p = probs + (size_t)row * V;
  const int base = part * kPart;
  uint64_t top[kTopK];
#pragma unroll
  for (int j = 0; j < kTopK; ++j) top[j] = 0;  // below every real key

  if ((V & 3) == 0 && (((uintptr_t)p) & 15) == 0) {
    const float4* p4 = (const float4*)(p + base);
    const int n4 = min(kPart, V - base) / 4;
    float4 x[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = tid + kThreads * u;
      x[u] = i < n4 ? p4[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = tid + kThreads * u;
      if (i < n4) {
        const int id = base + 4 * i;
        insert_key(top, rank_key(x[u].x, id));
        insert_key(top, rank_key(x[u].y, id + 1));
        insert_key(top, rank_key(x[u].z, id + 2));
        insert_key(top, rank_key(x[u].w, id + 3));
      }
    }
  } else {
    float x[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int i = base + tid + kThreads * u;
      x[u] = i < V ? p[i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int i = base + tid + kThreads * u;
      if (i < V) insert_key(top, rank_key(x[u], i));
    }
  }

  // Merge the 64 lists of each wave with shuffles, then the 4 wave lists.
  wave_merge_top8(top, 64);
  __shared__ uint64_t lists[kThreads / 64][kTopK];
  const int lane = tid & 63, wave = tid >> 6;
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < kTopK; ++j) lists[wave][j] = top[j];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int j = 0; j < kTopK; ++j) top[j] = lane < kThreads / 64 ? lists[lane][j] : 0;
  wave_merge_top8(top, kThreads / 64);
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < kTopK; ++j) lists[0][j] = top[j];
  }
  __builtin_amdgcn_wave_barrier();
  if (tid < kTopK) top_out[((size_t)row * P + part) * kTopK + tid] = lists[0][tid];
}

// S(p): 7, 5, 3, 1 on (0, 0.3], (0.3, 0.6], (0.6, 0.8], (0.8, 1].
__device__ __forceinline__ int expansion_size(float p) {
  if (p <= 0.3f) return 7;
  if (p <= 0.6f) return 5;
  if (p <= 0.8f) return 3;
  return 1;
}

// One workgroup per sequence.  First each wave merges the per-part top-8
// lists of its positions into one top-8 list per position (bitonic merges
// across lanes).  Then wave 0 assembles the tree: candidate c enumerates
// (position i, rank r) in linearisation order, and its confidence key is the
// top-8 key itself.
constexpr int kAsmThreads = 256;

__global__ __launch_bounds__(kAsmThreads) void cape_assemble(const uint64_t* __restrict__ part_top,
                                                             int gamma, int V, int k, int fixed,
                                                             int n_max, int32_t* __restrict__ tokens,
                                                             int32_t* __restrict__ parents,
                                                             int32_t* __restrict__ n_nodes) {
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int P = parts_per_row(V);
  const int C = P * kTopK;  // merge candidates per position

  __shared__ uint64_t top[kMaxNodes][kTopK];
  for (int i = wave; i < gamma; i += kAsmThreads / 64) {
    const uint64_t* src = part_top + ((size_t)b * gamma + i) * C;
    // Lane l holds the lists of parts l, l + 64, ...; fold them, then merge
    // across lanes.
    uint64_t best[kTopK];
#pragma unroll
    for (int j = 0; j < kTopK; ++j) best[j] = 0;
    for (int part = lane; part < P; part += 64) {
      uint64_t l[kTopK];
#pragma unroll
      for (int j = 0; j < kTopK; ++j) l[j] = src[part * kTopK + j];
      merge_top8(best, l);
    }
    int width = 1;
    while (width < min(P, 64)) width <<= 1;
    wave_merge_top8(best, width);
    if (lane == 0) {
#pragma unroll
      for (int j = 0; j < kTopK; ++j) top[i][j] = best[j];
    }
  }
  __syncthreads();
  if (wave != 0) return;

  __shared__ int sizes[kMaxNodes];
  __shared__ int base[kMaxNodes + 1];
  __shared__ uint64_t cand_key[kMaxNodes * 7];
  __shared__ int cand_pos[kMaxNodes * 7];

  if (lane < gamma) {
    const uint64_t k0 = top[lane][0];
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
  __builtin_amdgcn_wave_barrier();
  if (lane == 0) {
    int acc = 0;
    for (int i = 0; i < gamma; ++i) {
      base[i] = acc;
      acc += sizes[i];
    }
    base[gamma] = acc;
  }
  __builtin_amdgcn_wave_barrier();
  const int Ctot = base[gamma];
  for (int cidx = lane; cidx < Ctot; cidx += 64) {
    int i = 0;
    while (base[i + 1] <= cidx) ++i;
    const int r = cidx - base[i] + 1;
    cand_key[cidx] = top[i][r];
    cand_pos[cidx] = i;
  }
  __builtin_amdgcn_wave_barrier();

  const int budget = n_max - gamma;
  int written = 0;  // kept candidates in earlier chunks
  for (int cb = 0; cb < Ctot; cb += 64) {
    const int cidx = cb + lane;
    bool kept = false;
    if (cidx < Ctot) {
      if (Ctot <= budget) {
        kept = true;
      } else {
        // Rank in (prob desc, position asc, rank asc): probability is the
        // high half of the key; cidx order is (position, rank) order.
        const uint32_t pc = (uint32_t)(cand_key[cidx] >> 32);
        int ahead = 0;
        for (int o = 0; o < Ctot; ++o) {
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

size_t cape_workspace_bytes(int B, int gamma, int V) {
  return (size_t)B * gamma * ((V + kPart - 1) / kPart) * kTopK * sizeof(uint64_t);
}

hipError_t launch_cape_expand(const float* probs, int B, int gamma, int V, int k, int fixed,
                              int n_max, int32_t* tokens, int32_t* parents, int32_t* n_nodes,
                              void* ws, hipStream_t stream) {
  uint64_t* top = (uint64_t*)ws;
  const int P = (V + kPart - 1) / kPart;
  hipLaunchKernelGGL(cape_top8_part, dim3(P, B * gamma), dim3(kThreads), 0, stream, probs, V, top);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cape_assemble, dim3(B), dim3(kAsmThreads), 0, stream, top, gamma, V, k, fixed,
                     n_max, tokens, parents, n_nodes);
  return hipGetLastError();
}

}  // namespace glide
