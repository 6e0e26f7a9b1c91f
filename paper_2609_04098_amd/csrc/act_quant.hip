// Dynamic activation quantization to NVFP4 on gfx950 (paper, section 2
// "NVFP4"; the run-time "A4" half of W4A4).
//
// Two launches on the caller's stream (one for activations of at most 4096
// blocks, see act_quant_small_kernel), no atomics and no memset:
//   1. amax_partial: each workgroup reduces |x| over a grid-strided share of
//      X and writes one partial maximum to the workspace.  bf16 magnitudes
//      order like unsigned integers, so the reduction is packed u16 max.
//   2. quantize: every workgroup first reduces the partials to amax_X and
//      forms G = fl32(2688 / amax_X) (workgroup 0 writes it out), then each
//      thread quantizes 16-element blocks: 32 bytes of bf16 in, 8 bytes of
//      packed E2M1 codes and 1 byte of E4M3 scale out.
// In static mode pass 1 is skipped and G is read from the caller's scalar.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "launch.h"
#include "quant_device.h"

// Scratch memory of the allocation-free entry point
// (nvfp4_quantize_act_noalloc): the dynamic global scale's partial maxima,
// kActScratchBytes per device, held until the process ends.  Host code never
// uses this name as an address (it names a host-side stand-in); it takes the
// device address from hipGetSymbolAddress, once per device (act_scratch).
static __device__ __align__(256) float scratch[nvfp4::kActPartials];
static_assert(sizeof(scratch) == nvfp4::kActScratchBytes, "scratch size");

namespace nvfp4 {

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    uint32_t o = __shfl_xor(v, off, 64);
    v = v > o ? v : o;
  }
  return v;
}

__device__ __forceinline__ uint32_t block_max_u32(uint32_t v, uint32_t* lds) {
  v = wave_max_u32(v);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) lds[wave] = v;
  __syncthreads();
  uint32_t r = lds[0];
#pragma unroll
  for (int w = 1; w < kThreads / 64; ++w) r = r > lds[w] ? r : lds[w];
  __syncthreads();
  return r;
}

// Address of 16-byte vector `v` (8 bf16) of X: contiguous rows or stride ldx.
template <bool kContig>
__device__ __forceinline__ const uint4* vec_ptr(const uint16_t* x, uint32_t v, uint32_t vec_per_row,
                                                uint32_t ldx) {
  if (kContig) return reinterpret_cast<const uint4*>(x) + v;
  uint32_t row = v / vec_per_row, col = v - row * vec_per_row;
  return reinterpret_cast<const uint4*>(x + (size_t)row * ldx) + col;
}

template <bool kContig>
__global__ __launch_bounds__(kThreads) void amax_partial_kernel(const uint16_t* __restrict__ x,
                                                                uint32_t n_vec, uint32_t vec_per_row,
                                                                uint32_t ldx, float* __restrict__ partial) {
  __shared__ uint32_t lds[kThreads / 64];
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  u16x2 m = {0, 0};
  const uint32_t stride = gridDim.x * kThreads;
  uint32_t v = blockIdx.x * kThreads + threadIdx.x;
  // Four independent 16-byte loads in flight per thread.
  for (; v + 3 * stride < n_vec; v += 4 * stride) {
    uint4 d[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) d[u] = *vec_ptr<kContig>(x, v + u * stride, vec_per_row, ldx);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d[u].x & 0x7FFF7FFFu));
      m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d[u].y & 0x7FFF7FFFu));
      m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d[u].z & 0x7FFF7FFFu));
      m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d[u].w & 0x7FFF7FFFu));
    }
  }
  for (; v < n_vec; v += stride) {
    uint4 d = *vec_ptr<kContig>(x, v, vec_per_row, ldx);
    m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d.x & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d.y & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d.z & 0x7FFF7FFFu));
    m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d.w & 0x7FFF7FFFu));
  }
  uint32_t mx = m[0] > m[1] ? m[0] : m[1];
  mx = block_max_u32(mx, lds);
  if (threadIdx.x == 0) partial[blockIdx.x] = __uint_as_float(mx << 16);
}

// Grid-strided loop over 16-element blocks: 32 bytes of bf16 in, 8 bytes of
// packed codes and 1 scale byte out per block.  The next block's loads are
// issued before the current block is quantized (two blocks in flight per
// thread).  (Walking the blocks from the end of X to its start after the
// amax pass, so as to meet the most recently read part of X in the MALL,
// measured 2% slower on a 335 MB activation and is not done.)
template <bool kContig, bool kHuge>
__device__ __forceinline__ void quantize_blocks(const uint16_t* __restrict__ x, uint32_t n_blocks,
                                                uint32_t blocks_per_row, uint32_t ldx,
                                                uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                float g) {
  const float gd6 = g * (1.0f / 6.0f);
  const uint32_t stride = gridDim.x * kThreads;
  auto src_of = [&](uint32_t b) -> const uint4* {
    if (kContig) return reinterpret_cast<const uint4*>(x) + 2 * (size_t)b;
    const uint32_t row = b / blocks_per_row, col = b - row * blocks_per_row;
    return reinterpret_cast<const uint4*>(x + (size_t)row * ldx) + 2 * col;
  };
  uint32_t i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= n_blocks) return;
  const uint4* src = src_of(i);
  uint4 d0 = src[0], d1 = src[1];
  for (; i < n_blocks; i += stride) {
    const uint32_t b = i;
    uint4 e0 = d0, e1 = d1;
    if (i + stride < n_blocks) {
      const uint4* nxt = src_of(i + stride);
      e0 = nxt[0];
      e1 = nxt[1];
    }
    const uint32_t v[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
    uint32_t c0, c1;
    const uint32_t sc = quantize_block<kHuge>(v, g, gd6, c0, c1);
    reinterpret_cast<uint2*>(codes)[b] = make_uint2(c0, c1);
    scales[b] = (uint8_t)sc;
    d0 = e0;
    d1 = e1;
  }
}

template <bool kDynamic, bool kContig>
__global__ __launch_bounds__(kThreads) void act_quant_kernel(
    const uint16_t* __restrict__ x, uint32_t n_blocks, uint32_t blocks_per_row, uint32_t ldx,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, float* __restrict__ g_enc,
    const float* __restrict__ partial, uint32_t n_partial) {
  __shared__ uint32_t lds[kThreads / 64];
  float g;
  if (kDynamic) {
    uint32_t m = 0;
    for (uint32_t i = threadIdx.x; i < n_partial; i += kThreads) {
      uint32_t p = __float_as_uint(partial[i]);
      m = m > p ? m : p;                       // non-negative floats order as integers
    }
    g = global_scale(__uint_as_float(block_max_u32(m, lds)));
    if (blockIdx.x == 0 && threadIdx.x == 0) *g_enc = g;
  } else {
    g = *g_enc;
  }
  // The scale path is chosen per tensor, uniformly across the launch.
  if (g > kHugeScale)
    quantize_blocks<kContig, true>(x, n_blocks, blocks_per_row, ldx, codes, scales, g);
  else
    quantize_blocks<kContig, false>(x, n_blocks, blocks_per_row, ldx, codes, scales, g);
}

__global__ void write_zero_scale_kernel(float* g_enc) { *g_enc = 0.0f; }

// Small activations (decode-shaped calls, a few tokens): one workgroup does
// both passes, so the quantizer is one launch instead of two.  The amax is
// the same order-free maximum; the blocks are quantized by the same code.
constexpr int kSmallThreads = 1024;
// Up to 4096 blocks (M * K <= 65536, e.g. a few tokens of width 5120) one
// CU does the work faster than two launches spread over the chip.
constexpr uint32_t kSmallMaxBlocks = 4096;

template <bool kDynamic, bool kContig>
__global__ __launch_bounds__(kSmallThreads) void act_quant_small_kernel(
    const uint16_t* __restrict__ x, uint32_t n_blocks, uint32_t blocks_per_row, uint32_t ldx,
    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales, float* __restrict__ g_enc) {
  __shared__ uint32_t lds[kSmallThreads / 64];
  float g;
  if (kDynamic) {
    uint32_t m = 0;
    for (uint32_t b = threadIdx.x; b < n_blocks; b += kSmallThreads) {
      const uint4* src;
      if (kContig) {
        src = reinterpret_cast<const uint4*>(x) + 2 * (size_t)b;
      } else {
        uint32_t row = b / blocks_per_row, col = b - row * blocks_per_row;
        src = reinterpret_cast<const uint4*>(x + (size_t)row * ldx) + 2 * col;
      }
      const uint4 d0 = src[0], d1 = src[1];
      const uint32_t v[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
      const uint32_t a = __float_as_uint(block_amax(v));
      m = m > a ? m : a;
    }
    // Workgroup maximum (16 waves).
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) lds[threadIdx.x >> 6] = m;
    __syncthreads();
    m = lds[0];
#pragma unroll
    for (int w = 1; w < kSmallThreads / 64; ++w) m = m > lds[w] ? m : lds[w];
    g = global_scale(__uint_as_float(m));
    if (threadIdx.x == 0) *g_enc = g;
  } else {
    g = *g_enc;
  }
  const float gd6 = g * (1.0f / 6.0f);
  for (uint32_t b = threadIdx.x; b < n_blocks; b += kSmallThreads) {
    const uint4* src;
    if (kContig) {
      src = reinterpret_cast<const uint4*>(x) + 2 * (size_t)b;
    } else {
      uint32_t row = b / blocks_per_row, col = b - row * blocks_per_row;
      src = reinterpret_cast<const uint4*>(x + (size_t)row * ldx) + 2 * col;
    }
    const uint4 d0 = src[0], d1 = src[1];
    const uint32_t v[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
    uint32_t c0, c1, sc;
    if (g > kHugeScale)
      sc = quantize_block<true>(v, g, gd6, c0, c1);
    else
      sc = quantize_block<false>(v, g, gd6, c0, c1);
    reinterpret_cast<uint2*>(codes)[b] = make_uint2(c0, c1);
    scales[b] = (uint8_t)sc;
  }
}

static int grid_for(uint64_t work_items, int cap) {
  uint64_t g = (work_items + kThreads - 1) / kThreads;
  if (g > (uint64_t)cap) g = cap;
  return g < 1 ? 1 : (int)g;
}

hipError_t launch_act_amax(const void* x, int64_t M, int64_t K, int64_t ldx, float* partial, int* n_partial,
                           hipStream_t stream) {
  const bool contig = (ldx == K);
  const uint16_t* xp = static_cast<const uint16_t*>(x);
  const uint32_t n_vec = (uint32_t)(M * K / 8), vec_per_row = (uint32_t)(K / 8);
  *n_partial = grid_for(n_vec / 4, kActPartials);
  if (contig)
    hipLaunchKernelGGL(amax_partial_kernel<true>, dim3(*n_partial), dim3(kThreads), 0, stream, xp, n_vec,
                       vec_per_row, (uint32_t)ldx, partial);
  else
    hipLaunchKernelGGL(amax_partial_kernel<false>, dim3(*n_partial), dim3(kThreads), 0, stream, xp, n_vec,
                       vec_per_row, (uint32_t)ldx, partial);
  return hipGetLastError();
}

namespace {
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
float* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];
}  // namespace

hipError_t act_scratch(float** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  // Once per device, with that device current (the calling thread's).
  std::call_once(g_scratch_once[dev], [dev]() {
    void* p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = static_cast<float*>(p);
  });
  if (g_scratch_err[dev] != hipSuccess) return g_scratch_err[dev];
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_act_quant(const void* x, int64_t M, int64_t K, int64_t ldx, uint8_t* codes,
                            uint8_t* scales, float* g_enc, bool dynamic, float* partial,
                            hipStream_t stream) {
  if (M == 0 || K == 0) {
    if (dynamic) hipLaunchKernelGGL(write_zero_scale_kernel, dim3(1), dim3(1), 0, stream, g_enc);
    return hipGetLastError();
  }
  const bool contig = (ldx == K);
  const uint16_t* xp = static_cast<const uint16_t*>(x);
  const uint32_t n_vec = (uint32_t)(M * K / 8), vec_per_row = (uint32_t)(K / 8);
  const uint32_t n_blocks = (uint32_t)(M * K / 16), blocks_per_row = (uint32_t)(K / 16);
  if (n_blocks <= kSmallMaxBlocks) {
#define NVFP4_AQS(D, C)                                                                             \
  hipLaunchKernelGGL((act_quant_small_kernel<D, C>), dim3(1), dim3(kSmallThreads), 0, stream, xp, n_blocks, \
                     blocks_per_row, (uint32_t)ldx, codes, scales, g_enc)
    if (dynamic) {
      if (contig) NVFP4_AQS(true, true); else NVFP4_AQS(true, false);
    } else {
      if (contig) NVFP4_AQS(false, true); else NVFP4_AQS(false, false);
    }
#undef NVFP4_AQS
    return hipGetLastError();
  }
  int n_partial = 0;
  if (dynamic) {
    hipError_t e = launch_act_amax(x, M, K, ldx, partial, &n_partial, stream);
    if (e != hipSuccess) return e;
  }
  const int grid = grid_for(n_blocks, kActQuantGridCap);
#define NVFP4_AQ(D, C)                                                                          \
  hipLaunchKernelGGL((act_quant_kernel<D, C>), dim3(grid), dim3(kThreads), 0, stream, xp, n_blocks, \
                     blocks_per_row, (uint32_t)ldx, codes, scales, g_enc, partial, (uint32_t)n_partial)
  if (dynamic) {
    if (contig) NVFP4_AQ(true, true); else NVFP4_AQ(true, false);
  } else {
    if (contig) NVFP4_AQ(false, true); else NVFP4_AQ(false, false);
  }
#undef NVFP4_AQ
  return hipGetLastError();
}

}  // namespace nvfp4
