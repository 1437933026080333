// Projections of a few activation rows by a large weight matrix (arXiv
// 2402.02082, Sec. 4.1: the GliDe cross-attention sub-layer projects the
// draft's hidden rows into one query per target head, Q^{m,j} = H^m W_j, and
// the concatenated heads back, Concat(hd_1..hd_h) W^O).
//
//   out[m, n] = sum_k a[m, k] * w_t[n, k]      a [M, K], w_t [N, K] (bf16)
//
// With M <= 64 rows the weights dominate the bytes (every weight element is
// used M times), so the kernel streams w_t once: one workgroup per 16 output
// features, its four waves taking interleaved 32-wide K steps.  Each step is
// one v_mfma_f32_16x16x32_bf16 per 16-row tile of `a`, with A = 16 rows of
// w_t (16 contiguous bytes per lane) and B = the matching rows of `a` -- the
// same operand shapes as the attention kernel's K * Q^T.  Loads go through
// range-checked buffer descriptors (weight rows past N and activation rows
// past M read as zeros), eight steps in flight per wave in registers.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace glide {
namespace {

typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;

constexpr int kWaves = 4;
constexpr int kBufs = 8;             // K steps in flight per wave
constexpr uint32_t kDesc3 = 0x00020000u;
constexpr int kStream = 2;           // weights are read once: non-temporal
constexpr int kOutOfRange = 1 << 30; // past every descriptor (M * K * 2 < 2^30)

template <int AUX>
__device__ __forceinline__ u32x4_t load16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX));
}

template <int MT>
struct Step {
  u32x4_t w;
  u32x4_t a[MT];
};

template <int MT>
__device__ __forceinline__ void load_step(Step<MT>& s, __amdgpu_buffer_rsrc_t rw, __amdgpu_buffer_rsrc_t ra,
                                          int w_off, int a_off, int a_tile_stride, int kk, int K) {
  // kk: this lane's first k of the step; K % 8 == 0, so a lane's 8 values are
  // all inside the row or all past it.  Past it, the offset moves beyond
  // every descriptor's range, so the load returns zeros (no branch).
  const int kb = kk < K ? kk * 2 : kOutOfRange;
  s.w = load16<kStream>(rw, w_off + kb);
#pragma unroll
  for (int t = 0; t < MT; ++t) s.a[t] = load16<0>(ra, a_off + t * a_tile_stride + kb);
}

template <int MT>
__device__ __forceinline__ void mma_step(const Step<MT>& s, f32x4_t (&c)[MT]) {
#pragma unroll
  for (int t = 0; t < MT; ++t)
    c[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, s.w),
                                                  __builtin_bit_cast(bf16x8_t, s.a[t]), c[t], 0, 0, 0);
}

__device__ __forceinline__ void store_out(float* p, float v) { *p = v; }
__device__ __forceinline__ void store_out(uint16_t* p, float v) {
  *p = __builtin_bit_cast(uint16_t, (__bf16)v);
}

template <int MT, class OutT>
__global__ __launch_bounds__(64 * kWaves) void rows_matmul_kernel(const uint16_t* __restrict__ a,
                                                                  const uint16_t* __restrict__ w_t,
                                                                  OutT* __restrict__ out, int M,
                                                                  int K, int N) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int c = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16;
  // weight rows n0 .. n0 + 15 and activation rows 0 .. M - 1; rows past the
  // ends read as zeros
  const int w_rows = min(16, N - n0);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(w_t) + (size_t)n0 * K, (short)0, w_rows * K * 2, kDesc3);
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a), (short)0,
                                                                      M * K * 2, kDesc3);
  const int w_off = c * K * 2;       // A operand: weight row n0 + c
  const int a_off = c * K * 2;       // B operand: activation row 16 t + c
  const int a_tile_stride = 16 * K * 2;

  const int steps = (K + 31) / 32;
  const int my_steps = steps > wave ? (steps - wave + kWaves - 1) / kWaves : 0;
  const int iters = (my_steps + kBufs - 1) / kBufs;

  f32x4_t acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  Step<MT> buf[kBufs];
  int s = wave;  // this wave's steps: wave, wave + 4, ...
#pragma unroll
  for (int u = 0; u < kBufs; ++u)
    load_step<MT>(buf[u], rw, ra, w_off, a_off, a_tile_stride, 32 * (s + u * kWaves) + 8 * g, K);
  __builtin_amdgcn_sched_barrier(0);
  for (int it = 0; it + 1 < iters; ++it) {
#pragma unroll
    for (int u = 0; u < kBufs; ++u) {
      mma_step<MT>(buf[u], acc);
      load_step<MT>(buf[u], rw, ra, w_off, a_off, a_tile_stride, 32 * (s + kBufs * kWaves) + 8 * g, K);
      s += kWaves;
    }
  }
  if (iters > 0) {
#pragma unroll
    for (int u = 0; u < kBufs; ++u) mma_step<MT>(buf[u], acc);  // past-the-end steps are zeros
  }

  // Sum the four waves' partial products through LDS; wave 0 writes.
  __shared__ f32x4_t part[kWaves - 1][MT][64];
  if (wave > 0) {
#pragma unroll
    for (int t = 0; t < MT; ++t) part[wave - 1][t][lane] = acc[t];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int t = 0; t < MT; ++t) {
#pragma unroll
    for (int w = 0; w < kWaves - 1; ++w) acc[t] += part[w][t][lane];
    const int m = 16 * t + c;
    if (m < M) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = n0 + 4 * g + r;
        if (n < N) store_out(out + (size_t)m * N + n, acc[t][r]);
      }
    }
  }
}

template <class OutT>
hipError_t launch_rows(const uint16_t* a, const uint16_t* w_t, OutT* out, int M, int K, int N,
                       hipStream_t stream) {
  const dim3 grid((N + 15) / 16), block(64 * kWaves);
  const int mt = (M + 15) / 16;
  if (mt == 1)
    hipLaunchKernelGGL((rows_matmul_kernel<1, OutT>), grid, block, 0, stream, a, w_t, out, M, K, N);
  else if (mt == 2)
    hipLaunchKernelGGL((rows_matmul_kernel<2, OutT>), grid, block, 0, stream, a, w_t, out, M, K, N);
  else if (mt == 3)
    hipLaunchKernelGGL((rows_matmul_kernel<3, OutT>), grid, block, 0, stream, a, w_t, out, M, K, N);
  else
    hipLaunchKernelGGL((rows_matmul_kernel<4, OutT>), grid, block, 0, stream, a, w_t, out, M, K, N);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rows_matmul(const void* a, const void* w_t, void* out, int M, int K, int N,
                              bool out_bf16, hipStream_t stream) {
  // at most 64 activation rows per launch; more rows take further launches
  for (int m0 = 0; m0 < M; m0 += kMaxMatmulRows) {
    const int rows = min(kMaxMatmulRows, M - m0);
    const uint16_t* ap = (const uint16_t*)a + (size_t)m0 * K;
    hipError_t e = out_bf16
                       ? launch_rows(ap, (const uint16_t*)w_t, (uint16_t*)out + (size_t)m0 * N, rows, K, N, stream)
                       : launch_rows(ap, (const uint16_t*)w_t, (float*)out + (size_t)m0 * N, rows, K, N, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace glide
