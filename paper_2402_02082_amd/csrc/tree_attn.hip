// Split-K flash-decode attention of up to 64 query rows per (sequence, head)
// against a KV cache, for gfx950; and the block-masked cross attention of
// draft training, built from the same step.
//
// Computes hd = SoftMax(Q K^T * scale) V per head (arXiv 2402.02082, Sec. 4.1,
// MultiHead / hd_j equations).  In tree mode a query row (tree node n) sees
// the accepted prefix and the cache rows of its ancestor-or-self tree nodes,
// which is the CaPE verification mask (Sec. 4.2, mask_CaPE equation) for a
// linearised expanded proposal.  In cross mode (GliDe's cross-attention into
// the target cache, Sec. 4.1) every query row sees the prefix only.
//
// Work decomposition: one workgroup (4 waves) per (split, head, sequence).
// A split owns a contiguous key range, so every K/V byte is read from HBM
// once and is shared by all query rows of the sequence inside the MFMA tiles.
//  * Register kernel (bf16 with 1..16 rows, float32 with up to 64): the waves
//    take interleaved 32-key steps (16 for float32) with two steps of K/V in
//    flight per wave in registers.  Float32 with 17..32 rows gives each wave
//    both tiles; with 33..64 the waves form two groups of two, one per pair
//    of tiles (the second group's read of a step hits L2).
//  * Shared-step kernel (bf16 with 17..64 rows): each 32-key step goes from
//    HBM straight into an LDS ring, where every wave owning one of the
//    sequence's query tiles reads it.
//
// Per step and wave (bf16):
//   S^T[key, query] = K Q^T   on v_mfma_f32_16x16x32_bf16, A = 16 key rows
//                    (each lane holds 16 contiguous bytes of one key row),
//                    B = the resident Q fragments;
//   online softmax on S^T: the output layout puts one query per lane column,
//                    so the running max/sum are per-lane scalars; the
//                    reference max moves lazily, and only when it moves do the
//                    four 16-lane groups exchange their max (two row swaps);
//   O^T[d, query] += V^T P^T  on the same instruction, A = V^T built in
//                    registers: each lane holds 16 contiguous bytes (8 head
//                    dims) of 8 key rows and transposes the 8x8 block with
//                    byte permutes, B = P^T straight from the S^T registers.
// Tree masking is only evaluated in steps that reach the tree rows, from a
// 64-bit ancestor mask per query built by pointer doubling over the parents.
//
// The waves merge their (max, sum, O) states through LDS.  With more than one
// split per (sequence, head) each workgroup writes a partial state; for a
// single sequence it then counts itself in with one device-scope atomic,
// and the workgroup that completes the head merges the partials in split
// order -- one launch per call.  Calls with several sequences (and the
// shared-step kernel) leave the merge to a second small kernel.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "attn.h"

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
// Reductions over the four 16-lane groups of a wave (lanes c, c+16, c+32,
// c+48) with the gfx950 row-swap instructions: permlane16_swap(x, x) returns
// rows (0, 0, 2, 2) and (1, 1, 3, 3) of x, permlane32_swap(x, x) halves
// (0, 0) and (1, 1).  VALU only -- a lane shuffle through LDS would put an
// LDS round trip on the softmax's critical path.  Same pairing (and so the
// same float sums) as butterfly shuffles with lane offsets 16 and 32.
__device__ __forceinline__ float max_across_groups(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float sum_across_groups(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = __shfl((uint32_t)v, src);
  uint32_t hi = __shfl((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

// Ancestor-or-self bitmask of node `lane` (bit m set iff tree node m is the
// node itself or one of its ancestors), from that node's parent index.
// Pointer doubling: after round r the mask covers ancestors closer than 2^r
// and `p` points 2^r levels up; six rounds cover any depth <= 64.  Parents
// outside [-1, lane) count as -1.
__device__ __forceinline__ uint64_t ancestor_mask_from(int p, int N, int lane) {
  uint64_t a = 0;
  if (lane < N) {
    if (p < -1 || p >= lane) p = -1;
    a = 1ull << lane;
  } else {
    p = -1;
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

// K/V rows are fetched with buffer loads.  For each step the descriptor
// starts at the step's first key row and ends at the split's last key, so
// rows past the split read as zeros without touching memory (the partial
// last step and padding steps need no clamping and never see other splits'
// or uninitialised rows), the per-lane offsets stay fixed for the whole loop
// and the per-step part of the address lives in scalar registers.
// Word 3 of a gfx9 buffer descriptor: data format 32 bits (bits 15..18 = 4),
// no swizzle, raw (unstrided) addressing.
constexpr int kBufferDesc3 = 0x00020000;

// The range is a 32-bit unsigned byte count: at most 2^22 rows of 512 bytes
// (float32), i.e. 2^31, which the descriptor field holds but an int does not,
// so it is formed unsigned and passed on as the same bits.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t step_rsrc(const char* slab, int j0, int k_end,
                                                            int row_bytes) {
  const uint32_t rows = (uint32_t)max(k_end - j0, 0);
  const uint32_t range = rows * (uint32_t)row_bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(slab) + (size_t)j0 * row_bytes,
                                           (short)0, __builtin_bit_cast(int, range), kBufferDesc3);
}

// Cache policy of the K/V loads: kStream marks them non-temporal (each row is
// read once), which streams measurably faster when every K/V byte is
// fetched by one wave; kKeep leaves the default policy for kernels whose
// second query group re-reads each step from L2.
constexpr int kKeep = 0;
constexpr int kStream = 2;  // nt

template <int CPOL>
__device__ __forceinline__ u32x4_t load16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CPOL));
}

// Per-lane byte offsets inside one step, fixed for the whole loop.
struct LaneOffsets {
  int k0, k1;  // K rows
  int v0, v1;  // V rows
};

// bf16 (row = 256 bytes).  K: lane (c, g) reads rows 16*kt + c at bytes
// 64*st + 16*g; V: rows key_slot(g, i) = 16*(i / 4) + 4*g + i % 4 at 16*c.
__device__ __forceinline__ LaneOffsets lane_offsets(Bf16Path, int c, int g) {
  return LaneOffsets{c * 256 + 16 * g, (16 + c) * 256 + 16 * g, (4 * g) * 256 + 16 * c,
                     (16 + 4 * g) * 256 + 16 * c};
}

template <int CPOL>
__device__ __forceinline__ void load_kv(Bf16Path::KV& f, const char* kslab, const char* vslab,
                                        int j0, int k_end, const LaneOffsets& o) {
  const __amdgpu_buffer_rsrc_t rk = step_rsrc(kslab, j0, k_end, 256);
  const __amdgpu_buffer_rsrc_t rv = step_rsrc(vslab, j0, k_end, 256);
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    f.k[0][st] = load16<CPOL>(rk, o.k0 + 64 * st);
    f.k[1][st] = load16<CPOL>(rk, o.k1 + 64 * st);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f.v[i] = load16<CPOL>(rv, o.v0 + 256 * i);
    f.v[4 + i] = load16<CPOL>(rv, o.v1 + 256 * i);
  }
}

// float32 (row = 512 bytes).  K: row c at bytes 128*g + 16*e; V: rows
// 4*g + r at bytes 32*c + 16*h.
__device__ __forceinline__ LaneOffsets lane_offsets(F32Path, int c, int g) {
  return LaneOffsets{c * 512 + 128 * g, 0, (4 * g) * 512 + 32 * c, 0};
}

template <int CPOL>
__device__ __forceinline__ void load_kv(F32Path::KV& f, const char* kslab, const char* vslab, int j0,
                                        int k_end, const LaneOffsets& o) {
  const __amdgpu_buffer_rsrc_t rk = step_rsrc(kslab, j0, k_end, 512);
  const __amdgpu_buffer_rsrc_t rv = step_rsrc(vslab, j0, k_end, 512);
#pragma unroll
  for (int e = 0; e < 8; ++e) f.k[e] = __builtin_bit_cast(f32x4_t, load16<CPOL>(rk, o.k0 + 16 * e));
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      f.v[r][h] = __builtin_bit_cast(f32x4_t, load16<CPOL>(rv, o.v0 + 512 * r + 16 * h));
}

// Online-softmax state of one 16-query tile for the lane's query column.
// The reference max `m` is moved lazily: only when a new score exceeds it
// by more than kRescaleSlack (log2 units) are the accumulators rescaled, so
// probabilities stay <= 2^kRescaleSlack and most steps skip the rescale.
constexpr float kRescaleSlack = 8.f;

struct SoftmaxState {
  float m;  // reference max of scaled scores (log2 units); -inf until a key is seen
  float l;  // sum of exp2(score - m) over this lane's keys
};

// Given the raw scores x[] of this lane's keys for one query tile (masked
// ones -inf), decide whether the wave moves its reference max, rescale if so,
// and turn x[] into probabilities exp2(x * scale_log2 - m).  The decision
// needs no exchange between lanes: the reference moves when some lane's
// largest scaled score passes it by more than kRescaleSlack, and only then
// is the max taken over the column's lane groups.  The max is taken over the
// rounded scaled scores themselves, so the largest score of a row gets
// probability exactly 1 when it sets the reference.  Returns true when the
// accumulators must be rescaled by `alpha`.
template <int NV>
__device__ __forceinline__ bool softmax_update(float (&x)[NV], SoftmaxState& st, float scale_log2,
                                               float& alpha) {
#pragma unroll
  for (int i = 0; i < NV; ++i) x[i] *= scale_log2;
  // NaN-propagating maximum (v_maximum3_f32): scores are never NaN, and
  // unlike fmaxf it needs no quieting of the MFMA results first.
  float mx = x[0];
#pragma unroll
  for (int i = 1; i < NV; ++i) mx = __builtin_elementwise_maximum(mx, x[i]);
  const bool move = __any(mx > st.m + kRescaleSlack);
  alpha = 1.f;
  if (move) {
    const float m_new = fmaxf(st.m, max_across_groups(mx));
    alpha = (m_new == neg_inf()) ? 1.f : fast_exp2(st.m - m_new);
    st.m = m_new;
    st.l *= alpha;
  }
  const float m_ref = (st.m == neg_inf()) ? 0.f : st.m;
#pragma unroll
  for (int i = 0; i < NV; ++i) x[i] = fast_exp2(x[i] - m_ref);
  return move;
}

template <int NT, bool TREE>
__device__ __forceinline__ bool visible(int j, int Lb, int k_end, int N, const uint64_t (&anc)[NT],
                                        int nt) {
  if (j >= k_end) return false;
  if (j < Lb) return true;
  if (!TREE) return false;
  const unsigned m = (unsigned)(j - Lb);
  return m < (unsigned)N && ((anc[nt] >> m) & 1ull);
}

// V^T operands of a step: tile t holds head dim 8*c + t of the 8 keys of
// this lane's k-slots, i.e. element t of each loaded 8-dim chunk, two keys
// per dword (one byte permute per dword).
__device__ __forceinline__ void transpose_v(const u32x4_t (&v)[8], u32x4_t (&vt)[8]) {
#pragma unroll
  for (int w = 0; w < 4; ++w)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t a = v[2 * e][w], b = v[2 * e + 1][w];
      vt[2 * w][e] = __builtin_amdgcn_perm(b, a, 0x05040100u);      // low halves
      vt[2 * w + 1][e] = __builtin_amdgcn_perm(b, a, 0x07060302u);  // high halves
    }
}

// One wave step: scores, softmax update, PV accumulation.
template <int NT, bool TREE>
__device__ __forceinline__ void step(const Bf16Path::KV& f, const Bf16Path::QFrag (&qf)[NT],
                                     SoftmaxState (&sm)[NT], f32x4_t (&acc)[NT][8], int j0, int Lb,
                                     int k_end, int N, const uint64_t (&anc)[NT], float scale_log2,
                                     int g) {
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

  u32x4_t vt[8];
  transpose_v(f.v, vt);

#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const bool need_mask = (j0 + 32 > min(Lb, k_end));
    float x[8];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = s[kt][nt][r];
        if (need_mask && !visible<NT, TREE>(j0 + 16 * kt + 4 * g + r, Lb, k_end, N, anc, nt)) v = neg_inf();
        x[4 * kt + r] = v;
      }
    float alpha;
    if (softmax_update<8>(x, sm[nt], scale_log2, alpha)) {
#pragma unroll
      for (int t = 0; t < 8; ++t) acc[nt][t] *= alpha;
    }
    u32x4_t pw;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      pw[e] = pack_bf16x2(x[2 * e], x[2 * e + 1]);
      psum += x[2 * e] + x[2 * e + 1];
    }
    sm[nt].l += psum;
#pragma unroll
    for (int t = 0; t < 8; ++t)
      acc[nt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vt[t]), as_bf16x8(pw), acc[nt][t],
                                                           0, 0, 0);
  }
}

template <int NT, bool TREE>
__device__ __forceinline__ void step(const F32Path::KV& f, const F32Path::QFrag (&qf)[NT],
                                     SoftmaxState (&sm)[NT], f32x4_t (&acc)[NT][8], int j0, int Lb,
                                     int k_end, int N, const uint64_t (&anc)[NT], float scale_log2,
                                     int g) {
  const bool need_mask = (j0 + 16 > min(Lb, k_end));
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
      float v = a[r];
      if (need_mask && !visible<NT, TREE>(j0 + 4 * g + r, Lb, k_end, N, anc, nt)) v = neg_inf();
      x[r] = v;
    }
    float alpha;
    if (softmax_update<4>(x, sm[nt], scale_log2, alpha)) {
#pragma unroll
      for (int t = 0; t < 8; ++t) acc[nt][t] *= alpha;
    }
    sm[nt].l += (x[0] + x[1]) + (x[2] + x[3]);
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

__device__ __forceinline__ void store_2(uint16_t* dst, float a, float b) {
  *(uint32_t*)dst = pack_bf16x2(a, b);
}

__device__ __forceinline__ void store_2(float* dst, float a, float b) { *(float2*)dst = make_float2(a, b); }

// Split partial states.  They are written and read with the device-scope
// cache policy (sc1: stores written through past the XCD's L2, loads served
// coherently), so the workgroup that merges a (sequence, head) sees the
// states of every split whichever XCD -- and so whichever of the eight L2s --
// wrote them: nothing depends on where the dispatcher places a workgroup.
// One descriptor pair covers one (sequence, head): splits * N rows, at most
// 64 * 64 * 512 bytes of outputs.
constexpr int kDeviceScope = 16;  // sc1
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;

struct PartialRefs {
  __amdgpu_buffer_rsrc_t o, ml;  // rows split * N + n: 128 floats / (max, sum)
};

__device__ __forceinline__ PartialRefs partial_refs(const AttnArgs& a, int b, int h) {
  const int rows = a.splits * a.N;
  const size_t first = ((size_t)b * a.H + h) * (size_t)rows;
  PartialRefs r;
  r.o = __builtin_amdgcn_make_buffer_rsrc(a.part_o + first * kD, (short)0, rows * kD * 4, kBufferDesc3);
  r.ml = __builtin_amdgcn_make_buffer_rsrc(a.part_ml + first, (short)0, rows * 8, kBufferDesc3);
  return r;
}

// `coherent`: device-scope stores for the in-kernel merge; the second-launch
// merge reads the states after a kernel boundary and takes plain stores.
template <int CPOL>
__device__ __forceinline__ void store_partial_row8_p(const PartialRefs& p, int row, int d, const float (&o)[8]) {
  const int off = (row * kD + d) * 4;
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, f32x4_t{o[0], o[1], o[2], o[3]}), p.o,
                                         off, 0, CPOL);
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, f32x4_t{o[4], o[5], o[6], o[7]}), p.o,
                                         off + 16, 0, CPOL);
}

__device__ __forceinline__ void store_partial_row8(const PartialRefs& p, int row, int d, const float (&o)[8],
                                                   bool coherent) {
  if (coherent)
    store_partial_row8_p<kDeviceScope>(p, row, d, o);
  else
    store_partial_row8_p<0>(p, row, d, o);
}

__device__ __forceinline__ void store_partial_ml(const PartialRefs& p, int row, float m, float l,
                                                 bool coherent) {
  const u32x2_t v = __builtin_bit_cast(u32x2_t, f32x2_t{m, l});
  if (coherent)
    __builtin_amdgcn_raw_buffer_store_b64(v, p.ml, row * 8, 0, kDeviceScope);
  else
    __builtin_amdgcn_raw_buffer_store_b64(v, p.ml, row * 8, 0, 0);
}

// fp16 split states (bf16 inputs, in-kernel merge): the normalised output
// o / L of a query row in half precision, rounded to nearest even (one
// conversion per pair): a value's error is at most 2^-11 of its size, a
// quarter of what the bf16 rounding of every probability already allows.
// Rows of a wave that holds a value fp16 cannot represent (|x| > 65504,
// infinities, NaN) are also written in float32 to the float32 state rows,
// and the wave sets its (split, wave) bit in the flag words of the head's
// counter slot; the merge reads those rows instead.
constexpr float kHalfMax = 65504.f;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2_t;

__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), f16x2_t));
}

__device__ __forceinline__ float2 unpack_f16x2(uint32_t w) {
  const f16x2_t h = __builtin_bit_cast(f16x2_t, w);
  const f32x2_t f = __builtin_convertvector(h, f32x2_t);
  return make_float2(f[0], f[1]);
}

// fp16 rows: one descriptor per (sequence, head), splits * N rows of 256 B.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t half_refs(const AttnArgs& a, int b, int h) {
  const int rows = a.splits * a.N;
  const size_t first = ((size_t)b * a.H + h) * (size_t)rows;
  return __builtin_amdgcn_make_buffer_rsrc(a.part_h + first * kD, (short)0, rows * kD * 2, kBufferDesc3);
}

__device__ __forceinline__ void store_half_row8(__amdgpu_buffer_rsrc_t r, int row, int d, const float (&o)[8]) {
  const u32x4_t w = {pack_f16x2(o[0], o[1]), pack_f16x2(o[2], o[3]), pack_f16x2(o[4], o[5]), pack_f16x2(o[6], o[7])};
  __builtin_amdgcn_raw_buffer_store_b128(w, r, (row * kD + d) * 2, 0, kDeviceScope);
}

// Called by every thread of a split's workgroup once its partial stores are
// issued.  Each wave waits until its stores have completed at device scope;
// then one thread counts the split in and publishes the answer in the LDS
// word `flag` (a word the caller has free: the shared-step kernel passes one
// inside its ring, whose 64 KB must not grow -- a byte more and only one
// workgroup fits on a CU).  Returns true in the workgroup that completes the
// (sequence, head) -- after resetting the counter for the next call -- and
// false in the others, which are done.
__device__ __forceinline__ bool last_to_arrive(unsigned* counter, int nsplit, int* flag) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned before = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool last = before == (unsigned)(nsplit - 1);
    if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *flag = last;
  }
  __syncthreads();
  return *flag != 0;
}

// Merge of the split partial states of (sequence b, head h) by the
// workgroup that finished last: thread t takes output row t / (128 / DPT)
// and DPT head dims; the splits are combined in split order, so the result
// does not depend on which workgroup merges.  (Rows of up to 2 * DPT
// queries: DPT = 8 for 16 rows, 16 for 32, 32 for 64.)
// States from float32 inputs are the unnormalised (max, sum, O) of the
// second-launch merge.  States from bf16 inputs hold o / L: fp16 rows,
// requested together with every split's (max, sum) and the head's flag
// words, then -- for the (split, wave) pieces flagged there -- float32 rows
// in a second round.  Each split then enters with weight 2^(m_s - M) L_s.
// The merging workgroup clears the flags it found set.
template <class P, int DPT, bool HALF>
__device__ __forceinline__ void merge_partials(const AttnArgs& a, int b, int h, int nsplit) {
  typedef typename P::elem_t elem_t;
  constexpr bool kHalf = HALF && std::is_same<P, Bf16Path>::value && DPT == 8;
  constexpr int kTPR = kD / DPT;                          // threads per row
  constexpr int kBatch = DPT == 8 ? 8 : (DPT == 16 ? 4 : 2);  // splits requested at once
  const int tid = threadIdx.x;
  const int n = tid / kTPR, d0 = DPT * (tid % kTPR);
  const PartialRefs p = partial_refs(a, b, h);
  // fp16 rows, and the head's flag words: a batch of 8 splits is one word
  // (bit 4 u + wave), so word s0 / 8 comes with the batch's requests.
  const __amdgpu_buffer_rsrc_t ph = kHalf ? half_refs(a, b, h) : p.o;
  const __amdgpu_buffer_rsrc_t pf = __builtin_amdgcn_make_buffer_rsrc(
      a.counters + ((size_t)b * a.H + h) * kCounterStride + 1, (short)0, kWideFlagWords * 4, kBufferDesc3);
  const int r = (d0 & 31) >> 3;  // the wave of the split that wrote these dims
  uint32_t flagged = 0;  // batches whose flag word was set (thread 0 clears them)
  if (n < a.N) {
    float M = neg_inf(), L = 0.f, o[DPT];
#pragma unroll
    for (int e = 0; e < DPT; ++e) o[e] = 0.f;
    for (int s0 = 0; s0 < nsplit; s0 += kBatch) {
      f32x2_t ml[kBatch];
      float x[kBatch][DPT];
      const uint32_t wide = kHalf ? __builtin_amdgcn_raw_buffer_load_b32(pf, (s0 / 8) * 4, 0, kDeviceScope) : 0u;
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int row = min(s0 + u, nsplit - 1) * a.N + n;
        ml[u] = __builtin_bit_cast(f32x2_t, __builtin_amdgcn_raw_buffer_load_b64(p.ml, row * 8, 0, kDeviceScope));
        if (kHalf) {
          const u32x4_t hv = __builtin_bit_cast(
              u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(ph, (row * kD + d0) * 2, 0, kDeviceScope));
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const float2 f = unpack_f16x2(hv[w]);
            x[u][2 * w] = f.x;
            x[u][2 * w + 1] = f.y;
          }
        } else {
#pragma unroll
          for (int q = 0; q < DPT / 4; ++q) {
            const f32x4_t v = __builtin_bit_cast(
                f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(p.o, (row * kD + d0 + 4 * q) * 4, 0, kDeviceScope));
#pragma unroll
            for (int e = 0; e < 4; ++e) x[u][4 * q + e] = v[e];
          }
        }
      }
      if (kHalf && wide != 0u) {  // rare: float32 rows of the flagged pieces
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          if (s0 + u < nsplit && ((wide >> (4 * u + r)) & 1u)) {
            const int row = (s0 + u) * a.N + n;
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              const f32x4_t v = __builtin_bit_cast(
                  f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(p.o, (row * kD + d0 + 4 * q) * 4, 0, kDeviceScope));
#pragma unroll
              for (int e = 0; e < 4; ++e) x[u][4 * q + e] = v[e];
            }
          }
        }
        flagged |= 1u << (s0 / 8);
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const bool valid = s0 + u < nsplit;
        const float mu = valid ? ml[u][0] : neg_inf();
        const float m_new = fmaxf(M, mu);
        const float al = (m_new == neg_inf()) ? 0.f : fast_exp2(M - m_new);
        const float f = (m_new == neg_inf()) ? 0.f : fast_exp2(mu - m_new);
        const float w = kHalf ? f * ml[u][1] : f;  // fp16 rows are normalised
        L = L * al + (valid ? f * ml[u][1] : 0.f);
#pragma unroll
        for (int e = 0; e < DPT; ++e) o[e] = o[e] * al + (valid ? w * x[u][e] : 0.f);
        M = m_new;
      }
    }
    const float inv = (L > 0.f) ? 1.f / L : 0.f;
    elem_t* dst = (elem_t*)a.out + (((size_t)b * a.N + n) * a.H + h) * kD + d0;
#pragma unroll
    for (int i = 0; i < DPT / 8; ++i) {
      const float rr[8] = {o[8 * i] * inv,     o[8 * i + 1] * inv, o[8 * i + 2] * inv, o[8 * i + 3] * inv,
                           o[8 * i + 4] * inv, o[8 * i + 5] * inv, o[8 * i + 6] * inv, o[8 * i + 7] * inv};
      store_row8(dst + 8 * i, rr);
    }
  }
  if (kHalf) {
    // every thread has read the flags; thread 0 (row 0, which every batch
    // passes through) clears the words it found set, for the next call
    __syncthreads();
    if (tid == 0)
      for (int k = 0; k < kWideFlagWords; ++k)
        if ((flagged >> k) & 1u) __builtin_amdgcn_raw_buffer_store_b32(0u, pf, k * 4, 0, kDeviceScope);
  }
}

// Sequence taken by workgroup row y.  When every workgroup covers a whole
// sequence (one split) and 2 <= B <= 64, the y-th longest (ties to the lower
// index): the grid, dispatched in linear order, then starts the longest
// sequences' workgroups first, on CUs of their own, and the shortest ones
// share CUs -- longest-first scheduling, which shortens the ragged tail
// (33B and long-context shapes: -6 %).  Otherwise sequence y.  Ranks of
// raw lengths form a permutation, so every sequence is still taken exactly
// once and the results do not depend on the order.
__device__ __forceinline__ int seq_of_row(const int32_t* seq_lens, int B, int splits, int y, int lane) {
  if (splits != 1 || B < 2 || B > 64) return y;
  const int len = lane < B ? seq_lens[lane] : 0;
  int rank = 0;
  for (int j = 0; j < B; ++j) {
    const int lj = __shfl(len, j);
    rank += (lj > len) || (lj == len && j < lane);
  }
  const uint64_t hit = __ballot(lane < B && rank == y);
  return __builtin_amdgcn_readfirstlane(__ffsll((long long)hit) - 1);
}

// Work of one wave: the query tiles it owns and the key steps it takes.
// QG query groups split the 16-row query tiles; the 4 / QG waves of a group
// interleave the key steps of the split, so each K/V step is loaded by one
// wave per group (QG = 2 loads it twice, the second time from L2).
template <class P, int NT, int QG, bool TREE>
struct WaveTask {
  static constexpr int kWavesPerGroup = kWaves / QG;
  static constexpr int kStride = P::kStep * kWavesPerGroup;
  // K/V steps in flight per wave: two.  With one query tile this fits in
  // 256 registers, so two waves share each SIMD (two workgroups per CU) and
  // hide each other's dependency stalls; two tiles need the full register
  // file (one wave per SIMD).
  static constexpr int kBufs = 2;
  static constexpr int kCpol = QG == 1 ? kStream : kKeep;
};

template <class P, int NT, int QG, bool TREE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(NT == 1 ? 2 : 1)))
void tree_attn_kernel(AttnArgs args) {
  typedef typename P::elem_t elem_t;
  typedef WaveTask<P, NT, QG, TREE> Task;
  constexpr int kStep = P::kStep;
  constexpr int kBufs = Task::kBufs;
  constexpr int kWpg = Task::kWavesPerGroup;
  constexpr int kStride = Task::kStride;

  const int tid = threadIdx.x, lane = tid & 63;
  const int h = blockIdx.x, s = blockIdx.z;
  const int b = seq_of_row(args.seq_lens, args.B, args.splits, blockIdx.y, lane);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 15, g = lane >> 4;
  const int qg = wave / kWpg, wig = wave % kWpg;  // query group, wave in group
  const int N = args.N, H = args.H, Lcap = args.L_cap;

  const size_t head_off = ((size_t)b * H + h) * (size_t)Lcap * kD;
  const char* kslab = (const char*)((const elem_t*)args.k + head_off);
  const char* vslab = (const char*)((const elem_t*)args.v + head_off);
  const elem_t* qp = (const elem_t*)args.q;
  const LaneOffsets lo = lane_offsets(P{}, c, g);

  // Everything that does not depend on the sequence length is requested at
  // once: the length itself, the parent links, the queries and -- assuming
  // the split is full -- the first kBufs K/V steps (rows below L_cap, so in
  // bounds).  The length only arrives with them, one round trip later.
  const int raw_len = args.seq_lens[b];
  int my_parent = -1;
  if (TREE && lane < N) my_parent = args.parents[(size_t)b * N + lane];
  typename P::QFrag qf[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = 16 * (qg * NT + nt) + c;
    load_q<P>(qf[nt], qp + (((size_t)b * N + min(n, N - 1)) * H + h) * kD, n < N, g);
  }
  const int k_begin = s * args.chunk;
  const int first = k_begin + kStep * wig;  // this wave's steps: first + i * kStride
  const int full_end = min(Lcap, k_begin + args.chunk);
  typename P::KV buf[kBufs];
#pragma unroll
  for (int u = 0; u < kBufs; ++u) load_kv<Task::kCpol>(buf[u], kslab, vslab, first + u * kStride, full_end, lo);
  __builtin_amdgcn_sched_barrier(0);

  const int Lb = min(max(raw_len, 0), TREE ? Lcap - N : Lcap);
  const int T = Lb + (TREE ? N : 0);  // keys visible to some query
  const int nsplit = max(1, (T + args.chunk - 1) / args.chunk);
  if (s >= nsplit) return;
  const int k_end = min(T, k_begin + args.chunk);
  const int nsteps = first < k_end ? (k_end - first + kStride - 1) / kStride : 0;
  if (k_end < full_end) {
    // The split ends inside the cache: fetch again so that rows past the
    // sequence (possibly never written) read as zeros.
#pragma unroll
    for (int u = 0; u < kBufs; ++u) load_kv<Task::kCpol>(buf[u], kslab, vslab, first + u * kStride, k_end, lo);
  }

  // Ancestor masks are only needed by the split that holds the tree rows.
  uint64_t anc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) anc[nt] = 0;
  if (TREE && k_end > Lb) {
    const uint64_t mine = ancestor_mask_from(my_parent, N, lane);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) anc[nt] = shfl_u64(mine, min(16 * (qg * NT + nt) + c, 63));
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

  // Main loop, unrolled over the buffers: consume buffer u, refill it with
  // the step kBufs ahead.  The trip count is rounded up to whole rounds of
  // kBufs steps so the body is straight-line code and every wait leaves the
  // other buffers' loads in flight; steps at or past k_end read zeros and
  // are fully masked (the last round skips them).
  const int iters = (nsteps + kBufs - 1) / kBufs;
  int j = first;
  for (int it = 0; it + 1 < iters; ++it) {
#pragma unroll
    for (int u = 0; u < kBufs; ++u) {
      step<NT, TREE>(buf[u], qf, sm, acc, j, Lb, k_end, N, anc, args.scale_log2, g);
      load_kv<Task::kCpol>(buf[u], kslab, vslab, j + kBufs * kStride, k_end, lo);
      j += kStride;
    }
  }
  // Last round without refills: a load issued past the final step would
  // only hold up the merge below, which must wait for its registers.
  if (iters > 0) {
#pragma unroll
    for (int u = 0; u < kBufs; ++u) {
      if (u == 0 || j < k_end) step<NT, TREE>(buf[u], qf, sm, acc, j, Lb, k_end, N, anc, args.scale_log2, g);
      j += kStride;
    }
  }

#pragma unroll
  for (int nt = 0; nt < NT; ++nt) sm[nt].l = sum_across_groups(sm[nt].l);

  // Merge the waves of each query group through LDS.  Every wave publishes
  // its (max, sum) and its O^T accumulators, then finishes 4 / kWpg of the
  // four dim blocks r (d = 32 g + 8 r + t) of the group's tiles from all
  // the group's states, so the merge and the stores are shared out instead
  // of left to one wave.  Lane-major float4 layout: conflict-free 16-byte
  // LDS accesses.  States are combined in wave order (results do not depend
  // on which wave finishes a block).
  constexpr int kRPerWave = 4 / kWpg;
  __shared__ f32x4_t lds_o[QG][kWpg][NT][4][2][64];
  __shared__ float lds_m[QG][kWpg][NT][64];
  __shared__ float lds_l[QG][kWpg][NT][64];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    lds_m[qg][wig][nt][lane] = sm[nt].m;
    lds_l[qg][wig][nt][lane] = sm[nt].l;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      lds_o[qg][wig][nt][r][0][lane] = f32x4_t{acc[nt][0][r], acc[nt][1][r], acc[nt][2][r], acc[nt][3][r]};
      lds_o[qg][wig][nt][r][1][lane] = f32x4_t{acc[nt][4][r], acc[nt][5][r], acc[nt][6][r], acc[nt][7][r]};
    }
  }
  // Split states merged inside the kernel (single sequence) from bf16
  // inputs are stored as o / L in fp16 (see store_half_row8).
  constexpr bool kHalfCapable = std::is_same<P, Bf16Path>::value && NT == 1 && QG == 1;
  const bool half_states = kHalfCapable && nsplit > 1 && args.counters != nullptr && args.part_h != nullptr;
  __syncthreads();

  const PartialRefs pr = partial_refs(args, b, h);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float mw[kWpg], fw[kWpg];
#pragma unroll
    for (int w = 0; w < kWpg; ++w) mw[w] = lds_m[qg][w][nt][lane];
    float M = mw[0];
#pragma unroll
    for (int w = 1; w < kWpg; ++w) M = fmaxf(M, mw[w]);
#pragma unroll
    for (int w = 0; w < kWpg; ++w) fw[w] = (M == neg_inf()) ? 0.f : fast_exp2(mw[w] - M);
    float L = fw[0] * lds_l[qg][0][nt][lane];
#pragma unroll
    for (int w = 1; w < kWpg; ++w) L += fw[w] * lds_l[qg][w][nt][lane];

    const int n = 16 * (qg * NT + nt) + c;
    const float inv = (nsplit == 1 || half_states) ? ((L > 0.f) ? 1.f / L : 0.f) : 1.f;
#pragma unroll
    for (int i = 0; i < kRPerWave; ++i) {
      const int r = wig * kRPerWave + i;
      f32x4_t lo4 = fw[0] * lds_o[qg][0][nt][r][0][lane], hi4 = fw[0] * lds_o[qg][0][nt][r][1][lane];
#pragma unroll
      for (int w = 1; w < kWpg; ++w) {
        lo4 += fw[w] * lds_o[qg][w][nt][r][0][lane];
        hi4 += fw[w] * lds_o[qg][w][nt][r][1][lane];
      }
      const float o[8] = {lo4[0] * inv, lo4[1] * inv, lo4[2] * inv, lo4[3] * inv,
                          hi4[0] * inv, hi4[1] * inv, hi4[2] * inv, hi4[3] * inv};
      const int d = 32 * g + 8 * r;
      if (half_states) {
        bool fits = true;
#pragma unroll
        for (int e = 0; e < 8; ++e) fits &= __builtin_fabsf(o[e]) <= kHalfMax;  // false for NaN too
        if (n < N) store_half_row8(half_refs(args, b, h), s * N + n, d, o);
        if (!__all(fits || n >= N)) {  // wave-uniform: rare
          if (n < N) store_partial_row8(pr, s * N + n, d, o, true);
          if (lane == 0) {
            const int bit = 4 * s + r;
            __hip_atomic_fetch_or(args.counters + ((size_t)b * H + h) * kCounterStride + 1 + (bit >> 5),
                                  1u << (bit & 31), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
        }
      } else if (n < N) {
        if (nsplit == 1)
          store_row8((elem_t*)args.out + (((size_t)b * N + n) * H + h) * kD + d, o);
        else
          store_partial_row8(pr, s * N + n, d, o, args.counters != nullptr);
      }
    }
    if (nsplit > 1 && n < N && g == 0 && wig == 0) store_partial_ml(pr, s * N + n, M, L, args.counters != nullptr);
  }
  __shared__ int lds_last;
  if (nsplit > 1 && args.counters &&
      last_to_arrive(args.counters + ((size_t)b * H + h) * kCounterStride, nsplit, &lds_last)) {
    if (half_states)
      merge_partials<P, 8 * NT * QG, true>(args, b, h, nsplit);
    else
      merge_partials<P, 8 * NT * QG, false>(args, b, h, nsplit);
  }
}

// ---------------------------------------------------------------------------
// Shared-step kernel for 17..64 query rows (bf16).  Each 32-key step is
// fetched once per workgroup, straight from HBM into an LDS ring (buffer
// loads with the `lds` modifier, against the same range-checked descriptors),
// and consumed there by every wave that owns one of the sequence's 16-row
// query tiles: with four tiles each wave owns one tile and walks every step;
// with two tiles two waves share a tile and take alternate steps.  A round
// is the set of steps the four waves consume together (one or two).  The
// ring holds kStages steps: while a round is read, the rest are in flight,
// and the loads of a round go out as soon as the round before it retires.
//
// LDS layout of one step: K rows then V rows, 32 rows x 256 B each, in
// 16-byte units.  K unit (row, chunk) sits at row * 16 + (chunk ^ (row & 15)),
// V unit (row, chunk) at row * 16 + chunk.  The loads write 64 consecutive
// units per instruction (four rows; K's chunks permuted), so each instruction
// still reads 1 KB of contiguous HBM.  The layouts are the ones gfx950's LDS
// reads without bank conflicts for the two operand patterns: K's reads take
// 16 rows of one chunk (conflicting 8-way unpermuted), V's take 16 chunks of
// one row for four rows (measured 2-way conflicting under K's permutation,
// conflict-free unpermuted).
//
// The compiler does not track LDS writes made by memory loads, so the ring
// is synchronised by hand: each wave waits for its own loads of round r
// (vmcnt) and a workgroup barrier publishes them and retires round r - 1,
// whose stage is then refilled.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int kStepBytes = 32 * 256 * 2;  // 32 keys of K and V (bf16)

// Wait until at most N of this wave's vector-memory operations are in
// flight, then meet the other waves -- without the release/acquire fences a
// __syncthreads() carries (for memory-to-LDS loads those fences wait for
// every outstanding load, which would drain the ring each round).  The
// memory clobbers keep the compiler from moving LDS accesses across either.
template <int N>
__device__ __forceinline__ void ring_wait_and_meet() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
  asm volatile("s_barrier" ::: "memory");
}

__device__ __forceinline__ int k_unit(int row, int chunk) { return row * 16 + (chunk ^ (row & 15)); }
__device__ __forceinline__ int v_unit(int row, int chunk) { return row * 16 + chunk; }

// Global-side byte offset of the 16-byte chunk that lane `lane` moves for
// row `row` of a step: the LDS-DMA writes lane l's 16 bytes to unit l of the
// instruction's 64, so K lanes fetch the chunk their unit holds.
__device__ __forceinline__ int dma_k_off(int row, int lane) { return row * 256 + 16 * ((lane & 15) ^ (row & 15)); }
__device__ __forceinline__ int dma_v_off(int row, int lane) { return row * 256 + 16 * (lane & 15); }

// K and V fragments of one step, read from its LDS copy (layouts as load_kv).
__device__ __forceinline__ void read_step(Bf16Path::KV& f, const char* stepk, int c, int g) {
  const char* stepv = stepk + kStepBytes / 2;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int st = 0; st < 4; ++st)
      f.k[kt][st] = *(const u32x4_t*)(stepk + 16 * k_unit(16 * kt + c, 4 * st + g));
#pragma unroll
  for (int i = 0; i < 8; ++i)
    f.v[i] = *(const u32x4_t*)(stepv + 16 * v_unit(Bf16Path::key_slot(g, i), c));
}

template <int TQ, int LDS_BYTES, bool TREE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2 * LDS_BYTES <= 163840 ? 2 : 1)))
void tree_attn_shared_kernel(AttnArgs args) {
  constexpr int kWpt = kWaves / TQ;                // waves per query tile
  constexpr int kStages = LDS_BYTES / kStepBytes;        // ring stages, one step each
  constexpr int kStepInstr = kStepBytes / 1024 / kWaves;  // 1 KB loads per wave per step
  constexpr int kRoundKeys = 32 * kWpt;                   // a round: kWpt steps
  static_assert(kStages >= 2 * kWpt && kStages * kStepBytes == LDS_BYTES, "ring of two rounds or more");
  __shared__ __attribute__((aligned(1024))) char ring[LDS_BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int h = blockIdx.x, s = blockIdx.z;
  const int b = seq_of_row(args.seq_lens, args.B, args.splits, blockIdx.y, lane);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 15, g = lane >> 4;
  const int tile = wave % TQ, phase = wave / TQ;
  const int N = args.N, H = args.H, Lcap = args.L_cap;

  const int Lb = min(max(args.seq_lens[b], 0), TREE ? Lcap - N : Lcap);
  const int T = Lb + (TREE ? N : 0);
  const int nsplit = max(1, (T + args.chunk - 1) / args.chunk);
  if (s >= nsplit) return;
  const int k_begin = s * args.chunk;
  const int k_end = min(T, k_begin + args.chunk);
  const int rounds = k_end > k_begin ? (k_end - k_begin + kRoundKeys - 1) / kRoundKeys : 0;

  const size_t head_off = ((size_t)b * H + h) * (size_t)Lcap * kD;
  const char* kslab = (const char*)((const uint16_t*)args.k + head_off);
  const char* vslab = (const char*)((const uint16_t*)args.v + head_off);

  int my_parent = -1;
  if (TREE && lane < N) my_parent = args.parents[(size_t)b * N + lane];
  const int n = 16 * tile + c;
  const bool tile_live = 16 * tile < N;
  Bf16Path::QFrag qf[1];
  load_q<Bf16Path>(qf[0], (const uint16_t*)args.q + (((size_t)b * N + min(n, N - 1)) * H + h) * kD,
                   n < N, g);

  // This wave's share of step t: instruction k moves 1 KB (rows 4i..4i+3 of
  // K or V, i = wave + 4 * (k & 1)) into stage t % kStages; lanes fetch their
  // unit's chunk so the swizzled layout lands in place.
  const int dma_row = 4 * wave + (lane >> 4);
  const int dma_off[2] = {dma_k_off(dma_row, lane), dma_v_off(dma_row, lane)};
  auto issue_step = [&](int t) {
    char* stage = ring + (t % kStages) * kStepBytes;
    const int j0 = k_begin + 32 * t;
#pragma unroll
    for (int k = 0; k < kStepInstr; ++k) {
      const int m = k / 2, hi = k & 1;
      const __amdgpu_buffer_rsrc_t rs = step_rsrc(m ? vslab : kslab, j0, k_end, 256);
      char* dst = stage + m * (kStepBytes / 2) + (wave + 4 * hi) * 1024;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_t)dst, 16, dma_off[m] + 4096 * hi, 0, 0,
                                               kStream);
    }
  };
  // Round r issues steps kStages - kWpt + kWpt * r + i (i < kWpt), into the
  // stages of round r - 1; the prologue issues the steps before those.
#pragma unroll
  for (int t = 0; t < kStages - kWpt; ++t) issue_step(t);

  uint64_t anc[1] = {0};
  if (TREE && k_end > Lb) anc[0] = shfl_u64(ancestor_mask_from(my_parent, N, lane), min(n, 63));

  SoftmaxState sm[1];
  sm[0].m = neg_inf();
  sm[0].l = 0.f;
  f32x4_t acc[1][8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[0][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int r = 0; r < rounds; ++r) {
    // this wave's loads of round r have landed (at most the steps issued
    // after it, kStages - 2 * kWpt of them, are pending); after the barrier
    // everyone's have, and round r - 1 is retired
    ring_wait_and_meet<(kStages - 2 * kWpt) * kStepInstr>();
#pragma unroll
    for (int i = 0; i < kWpt; ++i) issue_step(kStages - kWpt + kWpt * r + i);
    const int t = kWpt * r + phase;
    const int j0 = k_begin + 32 * t;
    if (tile_live && j0 < k_end) {
      Bf16Path::KV f;
      read_step(f, ring + (t % kStages) * kStepBytes, c, g);
      if (j0 + 32 > k_end) {
        // rows past the split were not written by this round's loads
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (j0 + Bf16Path::key_slot(g, i) >= k_end) f.v[i] = u32x4_t{0, 0, 0, 0};
      }
      step<1, TREE>(f, qf, sm, acc, j0, Lb, k_end, N, anc, args.scale_log2, g);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();  // the ring is free for the merge below
  sm[0].l = sum_across_groups(sm[0].l);

  // Waves sharing a tile merge through LDS; phase 0 finishes the tile.
  float* mo = (float*)ring;                      // [TQ][8][4][64]
  float* mm = mo + TQ * 8 * 4 * 64;              // [TQ][64]
  float* ml = mm + TQ * 64;
  if (kWpt > 1 && phase == 1) {
    mm[tile * 64 + lane] = sm[0].m;
    ml[tile * 64 + lane] = sm[0].l;
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) mo[((tile * 8 + t) * 4 + r) * 64 + lane] = acc[0][t][r];
  }
  if (kWpt > 1) __syncthreads();
  if (phase != 0 || !tile_live) return;
  float M = sm[0].m, f0 = 1.f, f1 = 0.f, L = sm[0].l;
  if (kWpt > 1) {
    const float m1 = mm[tile * 64 + lane];
    M = fmaxf(sm[0].m, m1);
    f0 = (M == neg_inf()) ? 0.f : fast_exp2(sm[0].m - M);
    f1 = (M == neg_inf()) ? 0.f : fast_exp2(m1 - M);
    L = f0 * sm[0].l + f1 * ml[tile * 64 + lane];
  }
  const float inv = (nsplit == 1) ? ((L > 0.f) ? 1.f / L : 0.f) : 1.f;
  const size_t part_base = (((size_t)b * H + h) * args.splits + s) * N;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float o[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      float v = f0 * acc[0][t][r];
      if (kWpt > 1) v += f1 * mo[((tile * 8 + t) * 4 + r) * 64 + lane];
      o[t] = v * inv;
    }
    if (n < N) {
      const int d = 32 * g + 8 * r;
      if (nsplit == 1)
        store_row8((uint16_t*)args.out + (((size_t)b * N + n) * H + h) * kD + d, o);
      else
        store_row8(args.part_o + (part_base + n) * kD + d, o);
    }
  }
  if (nsplit > 1 && n < N && g == 0) args.part_ml[part_base + n] = make_float2(M, L);
}

// Merges the split partial states of every (sequence, head) whose keys were
// divided, in a fixed split order (the result does not depend on timing).
// One wave per output row (sequence, query, head); each lane owns two head
// dims and requests kBatch splits' partials at a time (the plan's split
// count, up to 8, so no request is a repeat).
constexpr int kCombineRows = kWaves;  // rows per workgroup

template <class P, int kBatch>
__global__ __launch_bounds__(kThreads) void tree_attn_combine(AttnArgs args) {
  typedef typename P::elem_t elem_t;
  const int N = args.N, H = args.H, Lcap = args.L_cap;
  const int row = blockIdx.x * kCombineRows + (threadIdx.x >> 6);  // (b, n, h) in out order
  const int lane = threadIdx.x & 63;
  if (row >= args.B * N * H) return;
  const int h = row % H, n = (row / H) % N, b = row / (H * N);
  const bool tree = args.parents != nullptr;
  const size_t base = ((size_t)b * H + h) * args.splits * N + n;  // + sp * N
  // The sequence length and the first batch of partials are requested
  // together; partials past this sequence's split count get weight 0.
  const int raw_len = args.seq_lens[b];
  float2 ml[kBatch], ov[kBatch];
#pragma unroll
  for (int u = 0; u < kBatch; ++u) {
    const int sp = min(u, args.splits - 1);
    ml[u] = args.part_ml[base + (size_t)sp * N];
    ov[u] = *(const float2*)(args.part_o + (base + (size_t)sp * N) * kD + 2 * lane);
  }
  // Pin the batch's loads above the early return below: the compiler
  // otherwise sinks them past it, and the partials are only requested once
  // the length has arrived (two round trips instead of one).
#pragma unroll
  for (int u = 0; u < kBatch; ++u) asm volatile("" : "+v"(ml[u].x), "+v"(ml[u].y), "+v"(ov[u].x), "+v"(ov[u].y));
  const int Lb = min(max(raw_len, 0), tree ? Lcap - N : Lcap);
  const int T = Lb + (tree ? N : 0);
  const int nsplit = max(1, (T + args.chunk - 1) / args.chunk);
  if (nsplit == 1) return;  // written directly by the attention kernel
  float M = neg_inf(), L = 0.f, o0 = 0.f, o1 = 0.f;
  for (int s0 = 0;;) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const bool valid = s0 + u < nsplit;
      const float mu = valid ? ml[u].x : neg_inf();
      const float m_new = fmaxf(M, mu);
      const float a = (m_new == neg_inf()) ? 0.f : fast_exp2(M - m_new);
      const float f = (m_new == neg_inf()) ? 0.f : fast_exp2(mu - m_new);
      // select, not multiply: entries past nsplit may hold stale values
      L = L * a + (valid ? f * ml[u].y : 0.f);
      o0 = o0 * a + (valid ? f * ov[u].x : 0.f);
      o1 = o1 * a + (valid ? f * ov[u].y : 0.f);
      M = m_new;
    }
    s0 += kBatch;
    if (s0 >= nsplit) break;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int sp = min(s0 + u, nsplit - 1);
      ml[u] = args.part_ml[base + (size_t)sp * N];
      ov[u] = *(const float2*)(args.part_o + (base + (size_t)sp * N) * kD + 2 * lane);
    }
  }
  const float inv = (L > 0.f) ? 1.f / L : 0.f;
  store_2((elem_t*)args.out + (size_t)row * kD + 2 * lane, o0 * inv, o1 * inv);
}

// LDS rings of the shared-step kernel: four 16 KB steps, so two workgroups
// share a CU.  Rings past 80 KB hold one workgroup per CU and measured
// slower; a five-step ring helps only grids of at most one workgroup per CU.
constexpr int kSharedLds4 = 65536;
constexpr int kSharedLds2 = 65536;


// One 32-key step of the block-masked kernel for the wave's NT query tiles.
// That kernel is compute-bound (every step feeds 32 queries per wave) and
// its vector-ALU work competes with the MFMA products for issue, so the
// per-score vector work is cut down against the shared step:
//  * masking runs only in the steps that reach tile 0's limit (the
//    smallest, wave-uniform); each lane then masks against its own limit;
//  * the reference max moves only when some lane's scaled score passes it by
//    more than kRescaleSlack -- one compare per lane finds that, and only
//    then is the max exchanged between the lane groups;
//  * probabilities are exp2(score * scale_log2 - m) with one fused
//    multiply-add, and the row sum adds them in float32 (the PV product
//    takes them rounded to bfloat16; the difference is far below the
//    output's rounding);
//  * the masking and the rescale sit in one branch each for all tiles, so
//    the common path is one straight block the scheduler can interleave.
template <int NT>
__device__ __forceinline__ void block_step(const Bf16Path::KV& f, const Bf16Path::QFrag (&qf)[NT],
                                           SoftmaxState (&sm)[NT], f32x4_t (&acc)[NT][8], int j0,
                                           const int (&tile_lo)[NT], const int (&lim)[NT],
                                           float scale_log2, int g) {
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

  u32x4_t vt[8];
  transpose_v(f.v, vt);

  float x[NT][8];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) x[nt][4 * kt + r] = s[kt][nt][r];
  if (j0 + 32 > tile_lo[0]) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (j0 + 16 * kt + 4 * g + r >= lim[nt]) x[nt][4 * kt + r] = neg_inf();
  }
  float mxs[NT];
  bool mv[NT];
  bool any_move = false;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    // NaN-propagating maximum (v_maximum3_f32): scores are never NaN, and
    // unlike fmaxf it needs no quieting of the MFMA results first.
    const float mx = __builtin_elementwise_maximum(
        __builtin_elementwise_maximum(__builtin_elementwise_maximum(x[nt][0], x[nt][1]), x[nt][2]),
        __builtin_elementwise_maximum(
            __builtin_elementwise_maximum(__builtin_elementwise_maximum(x[nt][3], x[nt][4]), x[nt][5]),
            __builtin_elementwise_maximum(x[nt][6], x[nt][7])));
    mxs[nt] = mx * scale_log2;
    mv[nt] = __any(mxs[nt] > sm[nt].m + kRescaleSlack);
    any_move |= mv[nt];
  }
  if (any_move) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (mv[nt]) {
        const float m_new = fmaxf(sm[nt].m, max_across_groups(mxs[nt]));
        const float alpha = (m_new == neg_inf()) ? 1.f : fast_exp2(sm[nt].m - m_new);
        sm[nt].m = m_new;
        sm[nt].l *= alpha;
#pragma unroll
        for (int t = 0; t < 8; ++t) acc[nt][t] *= alpha;
      }
    }
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float neg_m = (sm[nt].m == neg_inf()) ? 0.f : -sm[nt].m;
    u32x4_t pw;
    float l = sm[nt].l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float p0 = fast_exp2(fmaf(x[nt][2 * e], scale_log2, neg_m));
      const float p1 = fast_exp2(fmaf(x[nt][2 * e + 1], scale_log2, neg_m));
      pw[e] = pack_bf16x2(p0, p1);
      l += p0 + p1;
    }
    sm[nt].l = l;
#pragma unroll
    for (int t = 0; t < 8; ++t)
      acc[nt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vt[t]), as_bf16x8(pw), acc[nt][t],
                                                           0, 0, 0);
  }
}

// ---------------------------------------------------------------------------
// Block-masked cross attention of draft training (Sec. 4.1, "Block-wise
// Attention Mask"): the query at position p sees the target's keys of the
// earlier blocks, [0, block * floor(p / block)).  One workgroup per (head,
// sequence, 64 * kNT query positions), kNT 16-position tiles per wave (each
// K/V step read out of LDS once feeds every tile's products), keys streamed
// through the same LDS ring as the shared-step kernel, workgroups with the
// most keys first.  Each lane (query) compares the keys against its own
// limit, in the steps that reach its tile's limits.
// ---------------------------------------------------------------------------
template <int kNT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kNT <= 2 ? 2 : 1)))
void block_attn_kernel(BlockAttnArgs args) {
  constexpr int kStages = kSharedLds4 / kStepBytes;
  constexpr int kStepInstr = kStepBytes / 1024 / kWaves;
  constexpr int kBlockRows = 16 * kNT * kWaves;  // query positions per workgroup
  __shared__ __attribute__((aligned(1024))) char ring[kSharedLds4];

  // Dispatch order.  Workgroups go to the eight XCDs round-robin by linear
  // id, and each XCD has its own L2.  All query blocks of a (sequence, head)
  // pair are mapped to one XCD, and each XCD takes its pairs four at a time,
  // every query block of the four (most keys first) before the next four:
  // the blocks of a pair start together and stream the same K/V rows in
  // step, while the order over blocks stays longest first.  (Any dispatch
  // order gives the same results; this one only keeps reuse in L2.)
  const int P = gridDim.x * gridDim.y, Z = gridDim.z;
  const int lin = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  int pair, zi;
  if (P % 32 == 0) {
    const int x = lin % 8, k = lin / 8;
    const int grp = k / (4 * Z), r = k % (4 * Z);
    zi = r / 4;
    pair = (4 * grp + r % 4) * 8 + x;
  } else {
    pair = blockIdx.x + gridDim.x * blockIdx.y;
    zi = blockIdx.z;
  }
  const int h = pair % args.H, b = pair / args.H;
  const int p0 = (Z - 1 - zi) * kBlockRows;  // most keys first
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int c = lane & 15, g = lane >> 4;
  const int T = args.T, H = args.H, Lcap = args.L_cap, blk = args.block;

  const int p_last = min(p0 + kBlockRows - 1, T - 1);
  const int k_end = blk * (p_last / blk);            // the workgroup's largest limit
  const int steps = (k_end + 31) / 32;
  int p[kNT], my_limit[kNT], tile_lo[kNT];
  bool live[kNT];
  Bf16Path::QFrag qf[kNT];
#pragma unroll
  for (int nt = 0; nt < kNT; ++nt) {
    const int row0 = p0 + 16 * (kNT * wave + nt);
    p[nt] = row0 + c;
    live[nt] = row0 < T;
    my_limit[nt] = p[nt] < T ? blk * (p[nt] / blk) : 0;  // keys [0, limit) are visible
    tile_lo[nt] = live[nt] ? blk * (row0 / blk) : 0;     // the tile's smallest limit
    load_q<Bf16Path>(qf[nt], (const uint16_t*)args.q + (((size_t)b * T + min(p[nt], T - 1)) * H + h) * kD,
                     p[nt] < T, g);
  }
  const bool any_live = live[0];  // tile 0 of a wave is live whenever tile 1 is

  const size_t head_off = ((size_t)b * H + h) * (size_t)Lcap * kD;
  const char* kslab = (const char*)((const uint16_t*)args.k + head_off);
  const char* vslab = (const char*)((const uint16_t*)args.v + head_off);

  const int dma_row = 4 * wave + (lane >> 4);
  const int dma_off[2] = {dma_k_off(dma_row, lane), dma_v_off(dma_row, lane)};
  auto issue_step = [&](int t, int stage_idx) {
    char* stage = ring + stage_idx * kStepBytes;
    const int j0 = 32 * t;
#pragma unroll
    for (int k = 0; k < kStepInstr; ++k) {
      const int m = k / 2, hi = k & 1;
      const __amdgpu_buffer_rsrc_t rs = step_rsrc(m ? vslab : kslab, j0, k_end, 256);
      char* dst = stage + m * (kStepBytes / 2) + (wave + 4 * hi) * 1024;
      // default cache policy: every K/V row is read again by the workgroups
      // of the head's later query blocks, and the non-temporal hint of the
      // decode kernels (1.5x the HBM reads here) would evict it from L2
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_t)dst, 16, dma_off[m] + 4096 * hi, 0, 0,
                                               kKeep);
    }
  };
#pragma unroll
  for (int t = 0; t < kStages - 1; ++t) issue_step(t, t);

  SoftmaxState sm[kNT];
  f32x4_t acc[kNT][8];
#pragma unroll
  for (int nt = 0; nt < kNT; ++nt) {
    sm[nt].m = neg_inf();
    sm[nt].l = 0.f;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[nt][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  // Unrolled over the ring, so every step's stage (and with it each LDS
  // read's address) is a compile-time offset from per-lane base registers.
  for (int t0 = 0; t0 < steps; t0 += kStages) {
#pragma unroll
    for (int u = 0; u < kStages; ++u) {
      const int t = t0 + u;
      if (t < steps) {
        ring_wait_and_meet<(kStages - 2) * kStepInstr>();
        issue_step(t + kStages - 1, (u + kStages - 1) % kStages);
        const int j0 = 32 * t;
        if (any_live) {
          Bf16Path::KV f;
          read_step(f, ring + u * kStepBytes, c, g);
          if (j0 + 32 > k_end) {
#pragma unroll
            for (int i = 0; i < 8; ++i)
              if (j0 + Bf16Path::key_slot(g, i) >= k_end) f.v[i] = u32x4_t{0, 0, 0, 0};
          }
          block_step<kNT>(f, qf, sm, acc, j0, tile_lo, my_limit, args.scale_log2, g);
        }
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
  for (int nt = 0; nt < kNT; ++nt) {
    const float L = sum_across_groups(sm[nt].l);
    const float inv = (L > 0.f) ? 1.f / L : 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float o[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) o[t] = acc[nt][t][r] * inv;
      if (p[nt] < T)
        store_row8((uint16_t*)args.out + (((size_t)b * T + p[nt]) * H + h) * kD + 32 * g + 8 * r, o);
    }
  }
}

template <class P, bool TREE>
hipError_t launch_nt(const AttnArgs& args, hipStream_t stream) {
  // Heads vary fastest and splits slowest: workgroups are handed to the XCDs
  // round-robin by linear id, so every split level spreads over all eight
  // XCDs, and the empty splits of short sequences sit at the end of the grid.
  const int tiles = (args.N + 15) / 16;
  // The in-kernel merge is taken by the register kernel only: on the
  // shared-step kernel (bf16, 17..64 rows) the device-scope state stores
  // slowed the streams still running (13B shape: 49.4 against 42.6 us per
  // call), so that kernel leaves the counters alone and writes plain
  // partial states.
  const bool shared_step = std::is_same<P, Bf16Path>::value && tiles > 1;
  AttnArgs a = args;
  if (shared_step) a.counters = nullptr;
  const dim3 grid(a.H, a.B, a.splits), block(kThreads);
  if (tiles == 1)
    hipLaunchKernelGGL((tree_attn_kernel<P, 1, 1, TREE>), grid, block, 0, stream, a);
  else if (std::is_same<P, Bf16Path>::value && tiles == 2)
    hipLaunchKernelGGL((tree_attn_shared_kernel<2, kSharedLds2, TREE>), grid, block, 0, stream, a);
  else if (std::is_same<P, Bf16Path>::value)
    hipLaunchKernelGGL((tree_attn_shared_kernel<4, kSharedLds4, TREE>), grid, block, 0, stream, a);
  else if (tiles == 2)
    hipLaunchKernelGGL((tree_attn_kernel<P, 2, 1, TREE>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((tree_attn_kernel<P, 2, 2, TREE>), grid, block, 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1 || a.counters) return e;
  const int rows = a.B * a.N * a.H;
  const dim3 cgrid((rows + kCombineRows - 1) / kCombineRows);
  if (a.splits <= 2)
    hipLaunchKernelGGL((tree_attn_combine<P, 2>), cgrid, block, 0, stream, a);
  else if (a.splits <= 4)
    hipLaunchKernelGGL((tree_attn_combine<P, 4>), cgrid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((tree_attn_combine<P, 8>), cgrid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace

// Relative cost of s splits: the grid runs in ceil(B*H*s / CUs) waves of
// workgroups, each 1/s of a sequence long, and every split adds its partial
// results (written once, read once by the merge) to the K/V stream.
static double split_cost(long bh, int s, int N, int L_cap) {
  const double kv = (double)L_cap * kHeadDim * 2 * 2;                // K and V, bf16
  const double part = (double)N * (kHeadDim + 2) * sizeof(float);  // one split's partials
  const double waves = (double)((bh * s + kNumCU - 1) / kNumCU);
  return waves / s * (1.0 + (s > 1 ? 2.0 * s * part / kv : 0.0));
}

AttnPlan plan_tree_attn(int B, int N, int H, int L_cap, int max_splits) {
  AttnPlan p{};
  const int keys = L_cap;  // upper bound on the keys any query sees
  const long bh = (long)B * H;
  int want;
  if (max_splits > 0) {
    want = max_splits;
  } else {
    // Split only where it balances the CUs clearly better (a fifth less
    // cost), taking the fewest splits that reach the best cost, and keep
    // at least kMinChunk keys per split.
    const int most = min(kMaxSplits, (keys + kMinChunk - 1) / kMinChunk);
    const double one = split_cost(bh, 1, N, L_cap);
    double best = one;
    want = 1;
    for (int s = 2; s <= most; ++s) {
      const double c = split_cost(bh, s, N, L_cap);
      if (c < best - 1e-9) best = c, want = s;
    }
    if (best > 0.8 * one) want = 1;
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
  const size_t units = (size_t)bh * p.splits * N;
  p.counters_off = 0;
  p.part_ml_off = kCounterBytes;
  p.part_o_off = (p.part_ml_off + units * sizeof(float2) + 255) & ~(size_t)255;
  p.ws_bytes = p.part_o_off + units * kHeadDim * sizeof(float);
  // The last split to arrive merges only for single-sequence calls: their
  // splits end together, when the streams are draining.  With several
  // sequences the splits end at different times, and their device-scope
  // state stores slow the streams of the workgroups still running (ragged
  // batch of four, 16 rows: 62.3 against 59.8 us per call with the second
  // launch; two equal sequences: 19.4 against 18.0 us).
  p.merge_in_kernel = B == 1 && bh <= kCounterSlots;
  // fp16 states (bf16 calls) pay from 8 query rows on: one 16-node layer
  // 13.0 -> 11.8 us, an 8-node one 11.8 -> 11.4 us; 5 rows gain nothing
  // (5-query cross layer) or lose (5-chain over 512 keys: 7.6 -> 8.0 us).
  p.half_states = p.merge_in_kernel && N >= 8;
  if (p.half_states) {
    p.part_h_off = (p.ws_bytes + 255) & ~(size_t)255;
    p.ws_bytes = p.part_h_off + units * kHeadDim * sizeof(uint16_t);
  }
  return p;
}

hipError_t launch_block_attn(const BlockAttnArgs& a, hipStream_t stream) {
  // Two tiles per wave halve the LDS reads per query; take them while the
  // grid still gives every CU two workgroups.
  const long wgs2 = (long)a.H * a.B * ((a.T + 127) / 128);
  if (wgs2 >= 2L * kNumCU) {
    hipLaunchKernelGGL(block_attn_kernel<2>, dim3(a.H, a.B, (a.T + 127) / 128), dim3(kThreads), 0, stream, a);
  } else {
    hipLaunchKernelGGL(block_attn_kernel<1>, dim3(a.H, a.B, (a.T + 63) / 64), dim3(kThreads), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_tree_attn(const AttnArgs& a, bool bf16, hipStream_t stream) {
  const bool tree = a.parents != nullptr;
  if (bf16) return tree ? launch_nt<Bf16Path, true>(a, stream) : launch_nt<Bf16Path, false>(a, stream);
  return tree ? launch_nt<F32Path, true>(a, stream) : launch_nt<F32Path, false>(a, stream);
}

}  // namespace glide
