// Verify commit (arXiv 2402.02082): greedy acceptance of the candidate tree
// followed by the KV cache commit.  Sec. 3: the first accepted proposal
// tokens plus one token of the target's own extend the prefix; Sec. 4.1:
// after a verification step only the accepted tokens' cache rows are kept;
// Sec. 4.2: a tree candidate is accepted when its whole root path is.
//
// Workgroups of four waves, a few hundred in all: each sequence's (layer,
// head) slabs are dealt out in contiguous ranges to its workgroups and
// round-robin to their waves.  Every wave first works out its sequence's
// acceptance (one lane per node, ancestor masks by pointer doubling -- a few
// dozen instructions, cheaper than a second launch), then moves the accepted
// path's K and V rows of each of its slabs to the rows right behind the
// prefix, 16 loads per matrix in flight across slabs.  The path's node at
// depth d + 1 sits at row L + n_{d+1} >= L + d, so a destination row is never
// the source of a deeper slot; a slab's slots are visited in order and all
// sources of a batch are loaded before its stores, so a destination that is
// the source of a shallower slot is read first.  Each slab is moved by
// exactly one wave.
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

__global__ __launch_bounds__(64 * kWaves) void verify_commit_kernel(CommitArgs args, int slabs_per_wg) {
  const int b = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
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

  // The prefix length the rows are moved at: with caches to commit, clamped
  // into [0, L_cap - N] like every other reader of the lengths, and the
  // committed length is that same clamped value plus the accepted count;
  // with no caches (layers == 0) there is no cache bound and the length is
  // taken as given.
  const int raw_len = args.seq_lens[b];
  const int L = args.layers > 0 ? min(max(raw_len, 0), args.L_cap - N) : raw_len;
  if (blockIdx.x == 0 && wave == 0) {
    if (lane == 0) {
      args.accept_len[b] = a;
      args.seq_lens_out[b] = L + a;
      if (args.last_node) args.last_node[b] = last;
      if (args.bonus) args.bonus[b] = ta[last + 1];
    }
    if (args.path) {
      if (on_path) args.path[(size_t)b * N + rank] = lane;
      if (lane >= a && lane < N) args.path[(size_t)b * N + lane] = -1;
    }
  }
  __syncthreads();
  if (a == 0 || args.layers == 0) return;

  const int H = args.H, R = args.row_bytes;     // 256 (bf16) or 512 (fp32)
  const int lanes_per_row = R / 16;
  const int rows_per_load = 64 / lanes_per_row;
  const int chunk = lane % lanes_per_row, q = lane / lanes_per_row;
  const int s_begin = blockIdx.x * slabs_per_wg;
  const int s_end = min(args.layers * H, s_begin + slabs_per_wg);
  const int w = __builtin_amdgcn_readfirstlane(wave);
  const int mine = s_end > s_begin + w ? (s_end - s_begin - w + kWaves - 1) / kWaves : 0;
  const int upr = (a + rows_per_load - 1) / rows_per_load;  // load units per slab

  // Units in order: this wave's j-th slab s_begin + w + kWaves * j, its rows
  // rg * rows_per_load .. + rows_per_load - 1 (this lane: + q).  The cursor
  // (j, rg, layer, h) is wave-uniform and advances without divisions; each
  // batch replays it for the stores.
  struct Cursor {
    int j, rg, layer, h;
  };
  Cursor cur{0, 0, (s_begin + w) / H, (s_begin + w) % H};
  auto advance = [&](Cursor& c) {
    if (++c.rg == upr) {
      c.rg = 0;
      ++c.j;
      c.h += kWaves;
      while (c.h >= H) {
        c.h -= H;
        ++c.layer;
      }
    }
  };
  auto row_offset = [&](const Cursor& c) {
    return (((size_t)b * H + c.h) * args.L_cap + L) * R + chunk * 16;
  };
  while (cur.j < mine) {
    u32x4_t kx[kIter], vx[kIter];
    const Cursor start = cur;
#pragma unroll
    for (int i = 0; i < kIter; ++i) {
      if (cur.j < mine) {
        const int d = cur.rg * rows_per_load + q;
        const int n = d < a ? node_of[wave][d] : d;
        if (n != d) {  // a path that starts down the chain keeps those rows in place
          const size_t off = row_offset(cur) + (size_t)n * R;
          kx[i] = *(const u32x4_t*)(args.k[cur.layer] + off);
          vx[i] = *(const u32x4_t*)(args.v[cur.layer] + off);
        }
        advance(cur);
      }
    }
    Cursor st = start;
#pragma unroll
    for (int i = 0; i < kIter; ++i) {
      if (st.j < mine) {
        const int d = st.rg * rows_per_load + q;
        const int n = d < a ? node_of[wave][d] : d;
        if (n != d) {
          const size_t off = row_offset(st) + (size_t)d * R;
          *(u32x4_t*)(args.k[st.layer] + off) = kx[i];
          *(u32x4_t*)(args.v[st.layer] + off) = vx[i];
        }
        advance(st);
      }
    }
  }
}

}  // namespace

hipError_t launch_verify_commit(const float* logits, int V, const CommitArgs& a, hipStream_t stream) {
  hipError_t e = launch_argmax_rows(logits, a.B * (a.N + 1), V, a.target_argmax, stream);
  if (e != hipSuccess) return e;
  // about 512 workgroups in all, each sequence's slabs in equal ranges
  const int slabs = a.layers * a.H;
  const int want = max(1, min(slabs, (512 + a.B - 1) / a.B));
  const int per_wg = slabs > 0 ? (slabs + want - 1) / want : 0;
  const int groups = per_wg > 0 ? (slabs + per_wg - 1) / per_wg : 1;
  hipLaunchKernelGGL(verify_commit_kernel, dim3(groups, a.B), dim3(64 * kWaves), 0, stream, a, per_wg);
  return hipGetLastError();
}

}  // namespace glide
