// Split-K flash-decode attention of up to 64 query rows per (sequence, head)
// against a KV cache, for gfx950.
//
// Computes hd = SoftMax(Q K^T * scale) V per head (arXiv 2402.02082, Sec. 4.1,
// MultiHead / hd_j equations).  In tree mode a query row (tree node n) sees
// the accepted prefix and the cache rows of its ancestor-or-self tree nodes,
// which is the CaPE verification mask (Sec. 4.2, mask_CaPE equation) for a
// linearised expanded proposal.  In cross mode (GliDe's cross-attention into
// the target cache, Sec. 4.1) every query row sees the prefix only.
//
// Work decomposition: one workgroup (4 waves) per (split, head, sequence).
// A split owns a contiguous key range; its waves take interleaved 32-key
// steps (16 for float32), so every K/V byte is read from HBM exactly once and
// is shared by all query rows of the sequence inside the MFMA tiles.
//
// Per step and wave (bf16):
//   S^T[key, query] = K Q^T   on v_mfma_f32_16x16x32_bf16, A = 16 key rows
//                    (each lane loads 16 contiguous bytes of one key row),
//                    B = the resident Q fragments;
//   online softmax on S^T: the output layout puts one query per lane column,
//                    so the running max/sum are per-lane scalars and only the
//                    four 16-lane groups exchange their max (two shuffles);
//   O^T[d, query] += V^T P^T  on the same instruction, A = V^T built in
//                    registers: each lane loads 16 contiguous bytes (8 head
//                    dims) of 8 key rows and transposes the 8x8 block with
//                    byte permutes, B = P^T straight from the S^T registers.
// Tree masking is only evaluated in steps that reach the tree rows, from a
// 64-bit ancestor mask per query built by pointer doubling over the parents.
//
// The four waves merge their (max, sum, O) states through LDS; with more than
// one split the workgroup writes a partial state, and the last workgroup of a
// (sequence, head) to finish (a device-scope counter) merges all partials in
// a fixed split order and resets the counter.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace glide {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

constexpr int kD = kHeadDim;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

__device__ __forceinline__ float neg_inf() { return -__builtin_huge_valf(); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Max over the four 16-lane groups that hold the same query column.
__device__ __forceinline__ float max_across_groups(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}

__device__ __forceinline__ float sum_across_groups(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = __shfl((uint32_t)v, src);
  uint32_t hi = __shfl((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

// Ancestor-or-self bitmask of node `lane` (bit m set iff tree node m is the
// node itself or one of its ancestors).  Pointer doubling: after round r the
// mask covers ancestors closer than 2^r and `p` points 2^r levels up; six
// rounds cover any depth <= 64.  Parents outside [-1, lane) count as -1.
__device__ __forceinline__ uint64_t ancestor_mask(const int32_t* parents_b, int N,
                                                  int lane) {
  int p = -1;
  uint64_t a = 0;
  if (lane < N) {
    p = parents_b[lane];
    if (p < -1 || p >= lane) p = -1;
    a = 1ull << lane;
  }
#pragma unroll
  for (int round = 0; round < 6; ++round) {
    const int src = p < 0 ? lane : p;
    const uint64_t a_up = shfl_u64(a, src);
    const int p_up = __shfl(p, src);
    if (p >= 0) {
      a |= a_up;
      p = p_up;
    }
  }
  return a;
}

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Element types ------------------------------------------------------------

struct Bf16Path {
  static constexpr int kStep = 32;  // keys per wave step
  typedef uint16_t elem_t;
  struct QFrag { u32x4_t v[4]; };  // d = 32*st + 8*g + (0..7)
  struct KV {
    u32x4_t k[2][4];  // key row j0 + 16*kt + c, d = 32*st + 8*g + (0..7)
    u32x4_t v[8];     // key row j0 + key_slot(g, i), d = 8*c + (0..7)
  };
  // Key held in MFMA k-slot i of lane group g, matching where S^T puts it:
  // slots 0..3 are rows 4g..4g+3 of key tile 0, slots 4..7 those of tile 1.
  __device__ static __forceinline__ int key_slot(int g, int i) {
    return (i < 4) ? 4 * g + i : 16 + 4 * g + (i - 4);
  }
};

struct F32Path {
  static constexpr int kStep = 16;
  typedef float elem_t;
  struct QFrag { f32x4_t v[8]; };  // d = 32*g + 4*e + (0..3)
  struct KV {
    f32x4_t k[8];     // key row j0 + c, d = 32*g + 4*e + (0..3)
    f32x4_t v[4][2];  // key row j0 + 4*g + r, d = 8*c + 4*h + (0..3)
  };
};

template <class P>
__device__ __forceinline__ void load_q(typename P::QFrag& f, const typename P::elem_t* qrow,
                                       bool valid, int g);

template <>
__device__ __forceinline__ void load_q<Bf16Path>(Bf16Path::QFrag& f, const uint16_t* qrow,
                                                 bool valid, int g) {
#pragma unroll
  for (int st = 0; st < 4; ++st)
    f.v[st] = valid ? *(const u32x4_t*)(qrow + 32 * st + 8 * g) : u32x4_t{0, 0, 0, 0};
}

template <>
__device__ __forceinline__ void load_q<F32Path>(F32Path::QFrag& f, const float* qrow, bool valid,
                                                int g) {
#pragma unroll
  for (int e = 0; e < 8; ++e)
    f.v[e] = valid ? *(const f32x4_t*)(qrow + 32 * g + 4 * e) : f32x4_t{0.f, 0.f, 0.f, 0.f};
}

__device__ __forceinline__ void load_kv(Bf16Path::KV& f, const uint16_t* kp, const uint16_t* vp,
                                        int j0, int kmax, int c, int g) {
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    const int row = min(j0 + 16 * kt + c, kmax);
#pragma unroll
    for (int st = 0; st < 4; ++st)
      f.k[kt][st] = *(const u32x4_t*)(kp + (size_t)row * kD + 32 * st + 8 * g);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = min(j0 + Bf16Path::key_slot(g, i), kmax);
    f.v[i] = *(const u32x4_t*)(vp + (size_t)row * kD + 8 * c);
  }
}

__device__ __forceinline__ void load_kv(F32Path::KV& f, const float* kp, const float* vp, int j0,
                                        int kmax, int c, int g) {
  const int krow = min(j0 + c, kmax);
#pragma unroll
  for (int e = 0; e < 8; ++e) f.k[e] = *(const f32x4_t*)(kp + (size_t)krow * kD + 32 * g + 4 * e);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = min(j0 + 4 * g + r, kmax);
#pragma unroll
    for (int h = 0; h < 2; ++h) f.v[r][h] = *(const f32x4_t*)(vp + (size_t)row * kD + 8 * c + 4 * h);
  }
}

// Online-softmax state of one 16-query tile for the lane's query column.
struct SoftmaxState {
  float m;  // running max of scaled scores (log2 units)
  float l;  // running sum of exp2(score - m) over this lane's keys
};

// Scores of one step for one query tile -> masked, scaled, exponentiated.
// x[] holds S^T values for keys key_of(idx) of this lane; returns the
// rescale factor of the accumulators and leaves probabilities in x[].
template <int NV>
__device__ __forceinline__ float softmax_step(float (&x)[NV], SoftmaxState& st) {
  float mx = x[0];
#pragma unroll
  for (int i = 1; i < NV; ++i) mx = fmaxf(mx, x[i]);
  mx = max_across_groups(mx);
  const float m_new = fmaxf(st.m, mx);
  const float m_ref = (m_new == neg_inf()) ? 0.f : m_new;
  const float alpha = fast_exp2(st.m - m_ref);
#pragma unroll
  for (int i = 0; i < NV; ++i) x[i] = fast_exp2(x[i] - m_ref);
  st.m = m_new;
  return alpha;
}

template <int NT, bool TREE>
__device__ __forceinline__ bool visible(int j, int Lb, int N, const uint64_t (&anc)[NT], int nt) {
  if (j < Lb) return true;
  if (!TREE) return false;
  const unsigned m = (unsigned)(j - Lb);
  return m < (unsigned)N && ((anc[nt] >> m) & 1ull);
}

// One wave step: scores, softmax update, PV accumulation.
template <int NT, bool TREE>
__device__ __forceinline__ void step(const Bf16Path::KV& f, const Bf16Path::QFrag (&qf)[NT],
                                     SoftmaxState (&sm)[NT], f32x4_t (&acc)[NT][8], int j0, int Lb,
                                     int N, const uint64_t (&anc)[NT], float scale_log2, int g) {
  f32x4_t s[2][NT];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4_t a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 4; ++st)
        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(f.k[kt][st]), as_bf16x8(qf[nt].v[st]),
                                                    a, 0, 0, 0);
      s[kt][nt] = a;
    }

  // V^T operands: tile t holds head dim 8*c + t of the 8 keys of this lane's
  // k-slots, i.e. element t of each loaded 8-dim chunk, two keys per dword.
  u32x4_t vt[8];
#pragma unroll
  for (int w = 0; w < 4; ++w)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t a = f.v[2 * e][w], b = f.v[2 * e + 1][w];
      vt[2 * w][e] = (a & 0xFFFFu) | (b << 16);
      vt[2 * w + 1][e] = (a >> 16) | (b & 0xFFFF0000u);
    }

  const bool need_mask = (j0 + 32 > Lb);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float x[8];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = s[kt][nt][r] * scale_log2;
        if (need_mask && !visible<NT, TREE>(j0 + 16 * kt + 4 * g + r, Lb, N, anc, nt)) v = neg_inf();
        x[4 * kt + r] = v;
      }
    const float alpha = softmax_step<8>(x, sm[nt]);
    u32x4_t pw;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      pw[e] = pack_bf16x2(x[2 * e], x[2 * e + 1]);
      psum += bf16_lo(pw[e]) + bf16_hi(pw[e]);
    }
    sm[nt].l = sm[nt].l * alpha + psum;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      acc[nt][t] *= alpha;
      acc[nt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vt[t]), as_bf16x8(pw), acc[nt][t],
                                                           0, 0, 0);
    }
  }
}

template <int NT, bool TREE>
__device__ __forceinline__ void step(const F32Path::KV& f, const F32Path::QFrag (&qf)[NT],
                                     SoftmaxState (&sm)[NT], f32x4_t (&acc)[NT][8], int j0, int Lb,
                                     int N, const uint64_t (&anc)[NT], float scale_log2, int g) {
  const bool need_mask = (j0 + 16 > Lb);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    f32x4_t a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        a = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[e][i], qf[nt].v[e][i], a, 0, 0, 0);
    float x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = a[r] * scale_log2;
      if (need_mask && !visible<NT, TREE>(j0 + 4 * g + r, Lb, N, anc, nt)) v = neg_inf();
      x[r] = v;
    }
    const float alpha = softmax_step<4>(x, sm[nt]);
    sm[nt].l = sm[nt].l * alpha + ((x[0] + x[1]) + (x[2] + x[3]));
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[nt][t] *= alpha;
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int t = 0; t < 8; ++t)
        acc[nt][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.v[r][t >> 2][t & 3], x[r], acc[nt][t],
                                                          0, 0, 0);
  }
}

// Output stores: lane (c, g) owns query column c of each tile and head dims
// d = 32*g + 8*r + t (t = 0..7) of accumulator element acc[nt][t][r].
__device__ __forceinline__ void store_row8(uint16_t* dst, const float (&o)[8]) {
  u32x4_t w;
#pragma unroll
  for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(o[2 * e], o[2 * e + 1]);
  *(u32x4_t*)dst = w;
}

__device__ __forceinline__ void store_row8(float* dst, const float (&o)[8]) {
  *(f32x4_t*)dst = f32x4_t{o[0], o[1], o[2], o[3]};
  *(f32x4_t*)(dst + 4) = f32x4_t{o[4], o[5], o[6], o[7]};
}

__device__ __forceinline__ void store_4(uint16_t* dst, f32x4_t o) {
  uint32_t w0 = pack_bf16x2(o[0], o[1]), w1 = pack_bf16x2(o[2], o[3]);
  *(uint2*)dst = make_uint2(w0, w1);
}

__device__ __forceinline__ void store_4(float* dst, f32x4_t o) { *(f32x4_t*)dst = o; }

template <class P, int NT, bool TREE>
__global__ __launch_bounds__(kThreads) void tree_attn_kernel(AttnArgs args) {
  typedef typename P::elem_t elem_t;
  constexpr int kStep = P::kStep;

  const int s = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 15, g = lane >> 4;
  const int N = args.N, H = args.H, Lcap = args.L_cap;

  const int Lb = min(max(args.seq_lens[b], 0), TREE ? Lcap - N : Lcap);
  const int T = Lb + (TREE ? N : 0);  // keys visible to some query
  const int nsplit = max(1, (T + args.chunk - 1) / args.chunk);
  if (s >= nsplit) return;
  const int k_begin = s * args.chunk;
  const int k_end = min(T, k_begin + args.chunk);
  const int kmax = max(T - 1, 0);

  const size_t head_off = ((size_t)b * H + h) * (size_t)Lcap * kD;
  const elem_t* kp = (const elem_t*)args.k + head_off;
  const elem_t* vp = (const elem_t*)args.v + head_off;
  const elem_t* qp = (const elem_t*)args.q;

  typename P::QFrag qf[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = 16 * nt + c;
    load_q<P>(qf[nt], qp + (((size_t)b * N + min(n, N - 1)) * H + h) * kD, n < N, g);
  }

  uint64_t anc[NT];
  if (TREE) {
    const uint64_t mine = ancestor_mask(args.parents + (size_t)b * N, N, lane);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) anc[nt] = shfl_u64(mine, min(16 * nt + c, 63));
  } else {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) anc[nt] = 0;
  }

  SoftmaxState sm[NT];
  f32x4_t acc[NT][8];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    sm[nt].m = neg_inf();
    sm[nt].l = 0.f;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[nt][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  // Main loop: each wave takes every kWaves-th step of the split; the next
  // step's K/V are requested before the current one is consumed.
  int j0 = k_begin + kStep * wave;
  if (j0 < k_end) {
    typename P::KV cur, nxt;
    load_kv(cur, kp, vp, j0, kmax, c, g);
    for (;;) {
      const int jn = j0 + kStep * kWaves;
      const bool more = jn < k_end;
      if (more) load_kv(nxt, kp, vp, jn, kmax, c, g);
      step<NT, TREE>(cur, qf, sm, acc, j0, Lb, N, anc, args.scale_log2, g);
      if (!more) break;
      cur = nxt;
      j0 = jn;
    }
  }

#pragma unroll
  for (int nt = 0; nt < NT; ++nt) sm[nt].l = sum_across_groups(sm[nt].l);

  // Merge the four waves' states through LDS (lane-major: conflict free).
  __shared__ float lds_o[(kWaves - 1) * NT * 8 * 4 * 64];
  __shared__ float lds_m[(kWaves - 1) * NT * 64];
  __shared__ float lds_l[(kWaves - 1) * NT * 64];
  __shared__ int lds_last;
  if (wave > 0) {
    const int w = wave - 1;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      lds_m[(w * NT + nt) * 64 + lane] = sm[nt].m;
      lds_l[(w * NT + nt) * 64 + lane] = sm[nt].l;
#pragma unroll
      for (int t = 0; t < 8; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) lds_o[(((w * NT + nt) * 8 + t) * 4 + r) * 64 + lane] = acc[nt][t][r];
    }
  }
  __syncthreads();

  if (wave == 0) {
    const size_t part_base = (((size_t)b * H + h) * args.splits + s) * N;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float mw[kWaves], fw[kWaves];
      mw[0] = sm[nt].m;
#pragma unroll
      for (int w = 1; w < kWaves; ++w) mw[w] = lds_m[((w - 1) * NT + nt) * 64 + lane];
      float M = mw[0];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) M = fmaxf(M, mw[w]);
#pragma unroll
      for (int w = 0; w < kWaves; ++w) fw[w] = (M == neg_inf()) ? 0.f : fast_exp2(mw[w] - M);
      float L = fw[0] * sm[nt].l;
#pragma unroll
      for (int w = 1; w < kWaves; ++w) L += fw[w] * lds_l[((w - 1) * NT + nt) * 64 + lane];

      const int n = 16 * nt + c;
      const float inv = (nsplit == 1) ? ((L > 0.f) ? 1.f / L : 0.f) : 1.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float o[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          float v = fw[0] * acc[nt][t][r];
#pragma unroll
          for (int w = 1; w < kWaves; ++w) v += fw[w] * lds_o[((((w - 1) * NT + nt) * 8 + t) * 4 + r) * 64 + lane];
          o[t] = v * inv;
        }
        if (n < N) {
          const int d = 32 * g + 8 * r;
          if (nsplit == 1)
            store_row8((elem_t*)args.out + (((size_t)b * N + n) * H + h) * kD + d, o);
          else
            store_row8(args.part_o + (part_base + n) * kD + d, o);
        }
      }
      if (nsplit > 1 && n < N && g == 0) args.part_ml[part_base + n] = make_float2(M, L);
    }
  }
  if (nsplit == 1) return;

  // Publish this split's partial state; the last split of (b, h) merges.
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const uint32_t prev = __hip_atomic_fetch_add(args.counters + (size_t)b * H + h, 1u,
                                                 __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    lds_last = (prev == (uint32_t)(nsplit - 1));
  }
  __syncthreads();
  if (!lds_last) return;
  __threadfence();

  const size_t bh_base = ((size_t)b * H + h) * args.splits;
  for (int item = tid; item < N * (kD / 4); item += kThreads) {
    const int n = item / (kD / 4), dq = item % (kD / 4);
    float M = neg_inf();
    for (int sp = 0; sp < nsplit; ++sp) M = fmaxf(M, args.part_ml[(bh_base + sp) * N + n].x);
    float L = 0.f;
    f32x4_t o = {0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < nsplit; ++sp) {
      const float2 ml = args.part_ml[(bh_base + sp) * N + n];
      const float f = (M == neg_inf()) ? 0.f : fast_exp2(ml.x - M);
      L += f * ml.y;
      o += f * *(const f32x4_t*)(args.part_o + ((bh_base + sp) * N + n) * kD + 4 * dq);
    }
    const float inv = (L > 0.f) ? 1.f / L : 0.f;
    store_4((elem_t*)args.out + (((size_t)b * N + n) * H + h) * kD + 4 * dq, o * inv);
  }
  if (tid == 0)
    __hip_atomic_store(args.counters + (size_t)b * H + h, 0u, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

template <class P, bool TREE>
hipError_t launch_nt(const AttnArgs& a, hipStream_t stream) {
  const dim3 grid(a.splits, a.H, a.B), block(kThreads);
  const int nt = (a.N + 15) / 16;
  switch (nt) {
    case 1: hipLaunchKernelGGL((tree_attn_kernel<P, 1, TREE>), grid, block, 0, stream, a); break;
    case 2: hipLaunchKernelGGL((tree_attn_kernel<P, 2, TREE>), grid, block, 0, stream, a); break;
    case 3: hipLaunchKernelGGL((tree_attn_kernel<P, 3, TREE>), grid, block, 0, stream, a); break;
    default: hipLaunchKernelGGL((tree_attn_kernel<P, 4, TREE>), grid, block, 0, stream, a); break;
  }
  return hipGetLastError();
}

}  // namespace

AttnPlan plan_tree_attn(int B, int N, int H, int L_cap, int max_splits) {
  AttnPlan p{};
  const int keys = L_cap;  // upper bound on the keys any query sees
  int want;
  if (max_splits > 0) {
    want = max_splits;
  } else {
    const long bh = (long)B * H;
    want = (int)((2L * kNumCU + bh - 1) / bh);          // about two workgroups per CU
    want = min(want, (keys + 255) / 256);               // at least ~256 keys each
  }
  want = max(1, min(want, kMaxSplits));
  int chunk = (keys + want - 1) / want;
  chunk = ((chunk + kChunkQuantum - 1) / kChunkQuantum) * kChunkQuantum;
  p.chunk = max(chunk, kChunkQuantum);
  p.splits = max(1, (keys + p.chunk - 1) / p.chunk);
  if (p.splits == 1) {
    p.ws_bytes = 0;
    return p;
  }
  const size_t units = (size_t)B * H * p.splits * N;
  p.part_o_off = 0;
  p.part_ml_off = ((units * kHeadDim * sizeof(float)) + 255) & ~(size_t)255;
  p.counter_off = (p.part_ml_off + units * sizeof(float2) + 255) & ~(size_t)255;
  p.ws_bytes = p.counter_off + (size_t)B * H * sizeof(uint32_t);
  return p;
}

hipError_t launch_tree_attn(const AttnArgs& a, bool bf16, hipStream_t stream) {
  const bool tree = a.parents != nullptr;
  if (bf16) return tree ? launch_nt<Bf16Path, true>(a, stream) : launch_nt<Bf16Path, false>(a, stream);
  return tree ? launch_nt<F32Path, true>(a, stream) : launch_nt<F32Path, false>(a, stream);
}

}  // namespace glide
