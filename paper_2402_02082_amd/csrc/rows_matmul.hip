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
// registers.  From 21 activation rows on, rows_matmul_lds_kernel stages the
// activations through LDS instead (see there).
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
      // Keep each refill right after the products that free its registers:
      // left alone, the scheduler sinks all refills below all products, and
      // every round then drains the wave's loads to zero before reissuing
      // them (5 rows, packed weights: 7.8 -> 7.2 us per 4096 x 4096 launch).
      __builtin_amdgcn_sched_barrier(0);
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

// From 21 activation rows: the activations are staged through LDS.
// Read as MFMA operands straight from a row-major matrix, every load
// instruction takes a 64-byte slice of 16 rows 2K bytes apart -- half of 16
// cache lines -- and a probe streaming the same 80 x 4096 block that way
// per workgroup ran 2.7 times slower than in 1 KB contiguous pieces.  So
// four loader waves copy a 256-wide K chunk of every row into LDS with
// memory-to-LDS loads (each instruction two rows' 512 contiguous bytes),
// double-buffered, and four compute waves read their activation operands
// from there while their weights stream into registers, eight steps per
// wave in flight.  Keeping the two streams in different waves keeps the
// activations' L2 hits from queueing behind the weights' HBM reads (a
// wave's loads complete in order).  The chunk's 16-byte pieces are stored
// XOR-swizzled by row (piece q of row r at position q ^ (r % 16)), so the
// 16 rows of an operand read hit 16 different bank groups.  Each compute
// wave still takes steps wave, wave + 4, ... in order and the waves' sums
// are added in wave order: the same sums as rows_matmul_kernel, bit for bit.
typedef __attribute__((address_space(3))) void* lds_ptr_t;
constexpr int kChunkK = 256;               // K values per staged chunk (512 bytes a row)
constexpr int kChunkSteps = kChunkK / 32;  // 8 MFMA steps, two per compute wave
// Weight chunks requested ahead (two fragments each per compute wave), and
// staged activation chunks; deeper settings (8 weight chunks, 3-4 staged
// chunks where LDS holds them) measured the same.
constexpr int kWChunksAhead = 4;
constexpr int kStages = 2;

template <int MT, class OutT, bool PACKED>
__global__ __launch_bounds__(128 * kWaves) void rows_matmul_lds_kernel(const uint16_t* __restrict__ a,
                                                                       const uint16_t* __restrict__ w_t,
                                                                       OutT* __restrict__ out, int M, int K,
                                                                       int N) {
  constexpr int kRows = 16 * MT;
  constexpr int kBuf = kRows * kChunkK * 2;   // bytes of one staged chunk
  constexpr int kInstr = kRows / 2 / kWaves;  // memory-to-LDS loads per loader wave per chunk
  constexpr int WA = kWChunksAhead, NB = kStages;
  constexpr int kWAhead = 2 * WA;             // weight fragments in flight per compute wave
  __shared__ __attribute__((aligned(1024))) char abuf[NB * kBuf];
  __shared__ f32x4_t part[kWaves - 1][MT][64];

  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const bool loader = wid >= kWaves;
  const int wave = wid % kWaves;  // compute wave, or loader index
  const int c = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16;
  const int w_rows = min(16, N - n0);
  const int k_steps = (K + 31) / 32;
  const int chunks = (K + kChunkK - 1) / kChunkK;
  const __amdgpu_buffer_rsrc_t rw = PACKED
      ? __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(w_t) + (size_t)blockIdx.x * k_steps * 512,
                                          (short)0, k_steps * 1024, kDesc3)
      : __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(w_t) + (size_t)n0 * K, (short)0,
                                          w_rows * K * 2, kDesc3);
  // rows past M and columns past K read as zeros
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a), (short)0,
                                                                      M * K * 2, kDesc3);
  // weight operand of step st for this lane (zeros past K)
  auto wload = [&](int st) {
    const int kk = 32 * st + 8 * g;
    const int off = kk < K ? (PACKED ? st * 1024 + 16 * lane : c * K * 2 + kk * 2) : kOutOfRange;
    return load16<kStream>(rw, off);
  };
  // a loader wave's part of chunk ch into buffer b: instruction i covers
  // rows 2i and 2i + 1, lane l piece (l % 32) ^ (r % 16) of row r = 2i + l / 32
  auto stage = [&](int ch, int b) {
#pragma unroll
    for (int j = 0; j < kInstr; ++j) {
      const int i = wave + kWaves * j;
      const int r = 2 * i + (lane >> 5);
      const int kk = ch * kChunkK + 8 * ((lane & 31) ^ (r & 15));
      const int off = kk < K ? (r * K + kk) * 2 : kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(abuf + b * kBuf + i * 1024), 16, off, 0, 0, 0);
    }
  };

  f32x4_t acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  u32x4_t wf[kWAhead];  // slot 2 (ch % WA) + h: step ch * 8 + wave + 4 h

  // Loader and compute waves run loops of their own that meet at the same
  // two barriers per chunk.  In one shared loop the compiler's wait
  // insertion merged the loaders' memory-to-LDS loads into the compute
  // waves' state and made them wait for every weight load at each chunk;
  // for the same reason the compute loop has no per-chunk conditions in its
  // steady part (a group of WA chunks at a time, then the remainder).
  if (loader) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
      if (b < chunks) stage(b, b);
    for (int ch = 0; ch < chunks; ++ch) {
      // chunk ch staged: wait for this wave's loads of it (only the next
      // chunk's may stay in flight), then meet the compute waves
      if (ch + 1 < chunks)
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kInstr) : "memory");
      else
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      asm volatile("s_barrier" ::: "memory");
      asm volatile("s_barrier" ::: "memory");  // every wave is done with buffer ch & 1
      if (ch + NB < chunks) stage(ch + NB, ch & 1);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kWAhead; ++i) wf[i] = wload((i / 2) * kChunkSteps + wave + kWaves * (i % 2));
    auto chunk = [&](int ch, int u) {
      asm volatile("s_barrier" ::: "memory");
      const char* buf = abuf + (ch & 1) * kBuf;
      // all of the chunk's operand reads first, so their LDS latencies
      // overlap (one wave per SIMD computes)
      u32x4_t av[2][MT];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int sq = 4 * (wave + kWaves * h) + g;  // piece of this lane's operand
#pragma unroll
        for (int t = 0; t < MT; ++t) av[h][t] = *(const u32x4_t*)(buf + (16 * t + c) * 512 + 16 * (sq ^ c));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int t = 0; t < MT; ++t)
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wf[2 * u + h]),
                                                          __builtin_bit_cast(bf16x8_t, av[h][t]), acc[t], 0, 0, 0);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) wf[2 * u + h] = wload((ch + WA) * kChunkSteps + wave + kWaves * h);
      asm volatile("s_barrier" ::: "memory");
    };
    int ch0 = 0;
    for (; ch0 + WA <= chunks; ch0 += WA) {
#pragma unroll
      for (int u = 0; u < WA; ++u) chunk(ch0 + u, u);
    }
#pragma unroll
    for (int u = 0; u + 1 < WA; ++u)
      if (ch0 + u < chunks) chunk(ch0 + u, u);
  }

  // Sum the four compute waves' partial products through LDS; wave 0 writes.
  if (!loader && wave > 0) {
#pragma unroll
    for (int t = 0; t < MT; ++t) part[wave - 1][t][lane] = acc[t];
  }
  __syncthreads();
  if (loader || wave != 0) return;
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
  const dim3 grid((N + 15) / 16), block(64 * kWaves), block_lds(128 * kWaves);
  const int mt = (M + 15) / 16;
  // Up to 20 rows the operands come straight from memory; from 21 rows the
  // activations are staged through LDS (K = N = 4096, packed weights: 17
  // rows 9.6 against 10.3 us staged, 24 rows 11.3 against 10.3, 32 rows
  // 13.1 against 10.4, 80 rows 25.6 against 14.4).  Both give the same sums.
  switch (mt) {
    case 1: hipLaunchKernelGGL((rows_matmul_kernel<1, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N); break;
    case 2:
      if (M > 20)
        hipLaunchKernelGGL((rows_matmul_lds_kernel<2, OutT, PACKED>), grid, block_lds, 0, stream, a, w_t, out, M, K, N);
      else
        hipLaunchKernelGGL((rows_matmul_kernel<2, OutT, PACKED>), grid, block, 0, stream, a, w_t, out, M, K, N);
      break;
    case 3: hipLaunchKernelGGL((rows_matmul_lds_kernel<3, OutT, PACKED>), grid, block_lds, 0, stream, a, w_t, out, M, K, N); break;
    case 4: hipLaunchKernelGGL((rows_matmul_lds_kernel<4, OutT, PACKED>), grid, block_lds, 0, stream, a, w_t, out, M, K, N); break;
    case 5: hipLaunchKernelGGL((rows_matmul_lds_kernel<5, OutT, PACKED>), grid, block_lds, 0, stream, a, w_t, out, M, K, N); break;
    case 6: hipLaunchKernelGGL((rows_matmul_lds_kernel<6, OutT, PACKED>), grid, block_lds, 0, stream, a, w_t, out, M, K, N); break;
    case 7: hipLaunchKernelGGL((rows_matmul_lds_kernel<7, OutT, PACKED>), grid, block_lds, 0, stream, a, w_t, out, M, K, N); break;
    default: hipLaunchKernelGGL((rows_matmul_lds_kernel<8, OutT, PACKED>), grid, block_lds, 0, stream, a, w_t, out, M, K, N); break;
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
