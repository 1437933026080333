// Projections of a few activation rows by a large weight matrix (arXiv
// 2402.02082, Sec. 4.1: the GliDe cross-attention sub-layer projects the
// draft's hidden rows into one query per target head, Q^{m,j} = H^m W_j, and
// the concatenated heads back, Concat(hd_1..hd_h) W^O).
//
//   out[m, n] = sum_k a[m, k] * w_t[n, k]      a [M, K], w_t [N, K] (bf16)
//
// With M <= 128 rows the weights dominate the bytes (every weight element is
// used M times), so the kernel streams w_t once: one workgroup per 16 output
// features, its four waves taking interleaved 32-wide K steps.  Each step is
// one v_mfma_f32_16x16x32_bf16 per 16-row tile of `a`, with A = 16 rows of
// w_t (16 contiguous bytes per lane) and B = the matching rows of `a` -- the
// same operand shapes as the attention kernel's K * Q^T.  Loads go through
// range-checked buffer descriptors (weight rows past N and activation rows
// past M read as zeros), five to eight steps in flight per wave in
// registers.
//
// An operand tile spans 16 weight rows, so from a row-major w_t each load
// instruction fetches 64 bytes from each of 16 rows K * 2 bytes apart.  The
// packed layout (pack_rows_weights_kernel) stores every (16-row tile,
// 32-wide K step) operand as one 1 KB block in lane order -- lane l holds
// row l % 16, k 8 * (l / 16) .. + 7 -- so the same registers arrive from one
// contiguous 1 KB read.  Packing is a one-time transformation of static
// weights; both layouts give bit-identical results.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace glide {
namespace {

typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;

constexpr int kWaves = 4;
// K steps in flight per wave: eight while a step's registers are small; a
// step of MT activation tiles holds (1 + MT) x 16 bytes per lane, so larger
// row counts keep fewer in flight (at most 256 registers: two waves per SIMD).
template <int MT>
constexpr int bufs_for() { return MT <= 4 ? 8 : (MT <= 6 ? 6 : 5); }
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

template <int MT, bool PACKED>
__device__ __forceinline__ void load_step(Step<MT>& s, __amdgpu_buffer_rsrc_t rw, __amdgpu_buffer_rsrc_t ra,
                                          int w_off, int a_off, int a_tile_stride, int step, int g, int K) {
  // kk: this lane's first k of the step; K % 8 == 0, so a lane's 8 values are
  // all inside the row or all past it.  Past it, the offset moves beyond
  // every descriptor's range, so the load returns zeros (no branch).
  const int kk = 32 * step + 8 * g;
  const int kb = kk < K ? kk * 2 : kOutOfRange;
  // packed: step `step` of the tile is the 1 KB block at step * 1024
  s.w = load16<kStream>(rw, PACKED ? (kk < K ? step * 1024 + w_off : kOutOfRange) : w_off + kb);
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

template <int MT, class OutT, bool PACKED>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(MT > 4 ? 2 : 1)))
void rows_matmul_kernel(const uint16_t* __restrict__ a,
                                                                  const uint16_t* __restrict__ w_t,
                                                                  OutT* __restrict__ out, int M,
                                                                  int K, int N) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int c = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16;
  // weight rows n0 .. n0 + 15 and activation rows 0 .. M - 1; rows past the
  // ends read as zeros
  const int w_rows = min(16, N - n0);
  const int k_steps = (K + 31) / 32;
  // row-major: rows n0 .. n0 + w_rows - 1; packed: the tile's k_steps blocks
  // (rows past N are zeros in the packed copy)
  const __amdgpu_buffer_rsrc_t rw = PACKED
      ? __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(w_t) + (size_t)blockIdx.x * k_steps * 512,
                                          (short)0, k_steps * 1024, kDesc3)
      : __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(w_t) + (size_t)n0 * K, (short)0,
                                          w_rows * K * 2, kDesc3);
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a), (short)0,
                                                                      M * K * 2, kDesc3);
  const int w_off = PACKED ? 16 * lane : c * K * 2;  // A operand: weight row n0 + c
  const int a_off = c * K * 2;       // B operand: activation row 16 t + c
  const int a_tile_stride = 16 * K * 2;

  constexpr int kBufs = bufs_for<MT>();
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
    load_step<MT, PACKED>(buf[u], rw, ra, w_off, a_off, a_tile_stride, s + u * kWaves, g, K);
  __builtin_amdgcn_sched_barrier(0);
  for (int it = 0; it + 1 < iters; ++it) {
#pragma unroll
    for (int u = 0; u < kBufs; ++u) {
      mma_step<MT>(buf[u], acc);
      load_step<MT, PACKED>(buf[u], rw, ra, w_off, a_off, a_tile_stride, s + kBufs * kWaves, g, K);
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

template <class OutT, bool PACKED>
hipError_t launch_rows(const uint16_t* a, const uint16_t* w_t, OutT* out, int M, int K, int N,
                       hipStream_t stream) {
  const dim3 grid((N + 15) / 16), block(64 * kWaves);
  const int mt = (M + 15) / 16;
  switch (mt) {
    case 1: hipLaunchKernelGGL((rows_matmul_kernel<1, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
    case 2: hipLaunchKernelGGL((rows_matmul_kernel<2, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
    case 3: hipLaunchKernelGGL((rows_matmul_kernel<3, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
    case 4: hipLaunchKernelGGL((rows_matmul_kernel<4, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
    case 5: hipLaunchKernelGGL((rows_matmul_kernel<5, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
    case 6: hipLaunchKernelGGL((rows_matmul_kernel<6, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
    case 7: hipLaunchKernelGGL((rows_matmul_kernel<7, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
    default: hipLaunchKernelGGL((rows_matmul_kernel<8, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
  }
  return hipGetLastError();
}

// One thread per 16-byte unit of the packed copy: unit u of tile t, step j
// is lane u % 64 of that step's operand -- row 16t + (u % 16), k
// 32j + 8 * (u % 64 / 16) .. + 7 of w_t, or zeros past N or K.
__global__ __launch_bounds__(256) void pack_rows_weights_kernel(const uint16_t* __restrict__ w_t,
                                                                uint16_t* __restrict__ packed, int K,
                                                                int N, long units) {
  const long u = (long)blockIdx.x * 256 + threadIdx.x;
  if (u >= units) return;
  const int k_steps = (K + 31) / 32;
  const int l = (int)(u % 64);
  const long blk = u / 64;  // tile * k_steps + step
  const int step = (int)(blk % k_steps);
  const long tile = blk / k_steps;
  const long row = tile * 16 + (l & 15);
  const int k0 = 32 * step + 8 * (l >> 4);
  u32x4_t v = {0, 0, 0, 0};
  if (row < N && k0 < K) v = *(const u32x4_t*)(w_t + row * K + k0);
  *(u32x4_t*)(packed + u * 8) = v;
}

}  // namespace

size_t packed_rows_weights_bytes(int K, int N) {
  return (size_t)((N + 15) / 16) * ((K + 31) / 32) * 1024;
}

hipError_t launch_pack_rows_weights(const void* w_t, void* packed, int K, int N, hipStream_t stream) {
  const long units = (long)(packed_rows_weights_bytes(K, N) / 16);
  hipLaunchKernelGGL(pack_rows_weights_kernel, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, stream,
                     (const uint16_t*)w_t, (uint16_t*)packed, K, N, units);
  return hipGetLastError();
}

hipError_t launch_rows_matmul(const void* a, const void* w, void* out, int M, int K, int N,
                              bool out_bf16, bool packed, hipStream_t stream) {
  // at most kMaxMatmulRows activation rows per launch; more rows take
  // further launches, each streaming the weights again
  for (int m0 = 0; m0 < M; m0 += kMaxMatmulRows) {
    const int rows = min(kMaxMatmulRows, M - m0);
    const uint16_t* ap = (const uint16_t*)a + (size_t)m0 * K;
    const uint16_t* wp = (const uint16_t*)w;
    hipError_t e;
    if (out_bf16) {
      uint16_t* op = (uint16_t*)out + (size_t)m0 * N;
      e = packed ? launch_rows<uint16_t, true>(ap, wp, op, rows, K, N, stream)
                 : launch_rows<uint16_t, false>(ap, wp, op, rows, K, N, stream);
    } else {
      float* op = (float*)out + (size_t)m0 * N;
      e = packed ? launch_rows<float, true>(ap, wp, op, rows, K, N, stream)
                 : launch_rows<float, false>(ap, wp, op, rows, K, N, stream);
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace glide
