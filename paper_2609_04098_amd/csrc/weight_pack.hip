// Weight quantization and prepack for the NVFP4 GEMM (offline step).
//
// Each fused segment (a separately calibrated linear module, paper section 6)
// is quantized under its own global scale G_s = fl32(2688 / amax_s), with the
// same block rule as the activations (paper, section 2).  The codes and block
// scales are written straight into the GEMM's tile layout (packed_layout.h).
//
// Launches: segment amax partials -> one-workgroup finalize (writes G_s) ->
// pack over the padded block grid (padding gets zero codes and scales).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"
#include "packed_layout.h"
#include "quant_device.h"

namespace nvfp4 {

constexpr int kPackThreads = 256;

struct SegTable {
  int n_seg;
  uint32_t off[9];
};

__device__ __forceinline__ int segment_of(const SegTable& t, uint32_t n) {
  int s = 0;
#pragma unroll
  for (int i = 1; i < 8; ++i) s += (i < t.n_seg && n >= t.off[i]) ? 1 : 0;
  return s;
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    uint32_t o = __shfl_xor(v, off, 64);
    v = v > o ? v : o;
  }
  return v;
}

__device__ __forceinline__ uint32_t wg_max(uint32_t v, uint32_t* lds) {
  v = wave_max(v);
  if ((threadIdx.x & 63) == 0) lds[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t r = lds[0];
#pragma unroll
  for (int w = 1; w < kPackThreads / 64; ++w) r = r > lds[w] ? r : lds[w];
  __syncthreads();
  return r;
}

// grid (kWeightPartials, n_seg): workgroup (p, s) reduces |w| over a strided
// share of segment s's 16-byte vectors.
__global__ __launch_bounds__(kPackThreads) void seg_amax_kernel(const uint16_t* __restrict__ w,
                                                               uint32_t vec_per_row, uint32_t ldw,
                                                               SegTable segs, float* __restrict__ partial) {
  __shared__ uint32_t lds[kPackThreads / 64];
  const int s = blockIdx.y;
  const uint32_t row0 = segs.off[s], rows = segs.off[s + 1] - segs.off[s];
  const uint32_t n_vec = rows * vec_per_row;
  uint32_t m = 0;
  for (uint32_t v = blockIdx.x * kPackThreads + threadIdx.x; v < n_vec; v += gridDim.x * kPackThreads) {
    uint32_t r = v / vec_per_row, c = v - r * vec_per_row;
    uint4 d = reinterpret_cast<const uint4*>(w + (size_t)(row0 + r) * ldw)[c];
    uint32_t a = (d.x & 0x7FFF7FFFu), b = (d.y & 0x7FFF7FFFu), e = (d.z & 0x7FFF7FFFu), f = (d.w & 0x7FFF7FFFu);
    uint32_t vals[8] = {a & 0xFFFFu, a >> 16, b & 0xFFFFu, b >> 16, e & 0xFFFFu, e >> 16, f & 0xFFFFu, f >> 16};
#pragma unroll
    for (int i = 0; i < 8; ++i) m = m > vals[i] ? m : vals[i];
  }
  m = wg_max(m, lds);
  if (threadIdx.x == 0) partial[s * gridDim.x + blockIdx.x] = __uint_as_float(m << 16);
}

__global__ __launch_bounds__(kPackThreads) void seg_finalize_kernel(const float* __restrict__ partial,
                                                                   int n_part, int n_seg,
                                                                   float* __restrict__ g_enc_seg) {
  __shared__ uint32_t lds[kPackThreads / 64];
  for (int s = 0; s < n_seg; ++s) {
    uint32_t m = 0;
    for (int i = threadIdx.x; i < n_part; i += kPackThreads) {
      uint32_t p = __float_as_uint(partial[s * n_part + i]);
      m = m > p ? m : p;
    }
    m = wg_max(m, lds);
    if (threadIdx.x == 0) g_enc_seg[s] = global_scale(__uint_as_float(m));
  }
}

__global__ __launch_bounds__(kPackThreads) void pack_kernel(const uint16_t* __restrict__ w, uint32_t N,
                                                           uint32_t kb_valid, uint32_t ldw, uint32_t kb_pad,
                                                           uint32_t n_blocks_pad, uint32_t kc_count,
                                                           SegTable segs,
                                                           const float* __restrict__ g_enc_seg,
                                                           uint8_t* __restrict__ packed, uint32_t scale_offset) {
  for (uint32_t b = blockIdx.x * kPackThreads + threadIdx.x; b < n_blocks_pad; b += gridDim.x * kPackThreads) {
    uint32_t n = b / kb_pad, kb = b - n * kb_pad;
    uint32_t c0 = 0, c1 = 0, sc = 0;
    if (n < N && kb < kb_valid) {
      float g = g_enc_seg[segment_of(segs, n)];
      const uint4* src = reinterpret_cast<const uint4*>(w + (size_t)n * ldw) + 2 * kb;
      uint4 d0 = src[0], d1 = src[1];
      uint32_t v[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
      // Static segment scales may be exceeded by the data; such elements
      // saturate.
      sc = g > kHugeScale ? quantize_block<true>(v, g, g * (1.0f / 6.0f), c0, c1)
                          : quantize_block<false>(v, g, g * (1.0f / 6.0f), c0, c1);
    }
    *reinterpret_cast<uint2*>(packed + packed_code_offset(n, kb, kc_count)) = make_uint2(c0, c1);
    packed[scale_offset + packed_scale_offset(n, kb, kc_count)] = (uint8_t)sc;
  }
}

__global__ __launch_bounds__(kPackThreads) void unpack_kernel(const uint8_t* __restrict__ packed, uint32_t N,
                                                             uint32_t kb_valid, uint32_t kc_count,
                                                             uint32_t scale_offset,
                                                             uint8_t* __restrict__ codes,
                                                             uint8_t* __restrict__ scales) {
  const uint32_t n_blocks = N * kb_valid;
  for (uint32_t b = blockIdx.x * kPackThreads + threadIdx.x; b < n_blocks; b += gridDim.x * kPackThreads) {
    uint32_t n = b / kb_valid, kb = b - n * kb_valid;
    uint2 c = *reinterpret_cast<const uint2*>(packed + packed_code_offset(n, kb, kc_count));
    reinterpret_cast<uint2*>(codes)[b] = c;
    scales[b] = packed[scale_offset + packed_scale_offset(n, kb, kc_count)];
  }
}

// ------------------------------------------------- fused-group harmonization
//
// Paper, section 6 ("Per-module calibration vs. fused-GEMM scaling"): the
// segments of a fused weight are rewritten to one shared global scale, the
// smallest positive encode-direction G_s (the largest-amax segment's), and
// each block scale S of segment s becomes RNE_E4M3(S * G_shared / G_s); the
// E2M1 codes stay.  This is an offline rewrite, so it decides in float64,
// where every compared product is exact: S * G_shared has at most 4 + 24
// significant bits, (v_c + v_c+1) * G_s at most 5 + 24.

// Value of a non-negative E4M3 code (0..126) in float64, exactly.
__device__ __forceinline__ double e4m3_f64(uint32_t c) {
  const uint32_t e = c >> 3, m = c & 7u;
  if (e == 0) return (double)m * 0x1p-9;
  return __longlong_as_double((long long)(((uint64_t)(e - 7u + 1023u) << 52) | ((uint64_t)m << 49)));
}

// E4M3 code of RNE(value(c) * gs / gd) for binary32 gs, gd > 0, ties to the
// even code, saturating at 448.
__device__ __forceinline__ uint32_t fold_scale_code(uint32_t c, double gs, double gd) {
  const double num = e4m3_f64(c) * gs;
  uint32_t lo = 0, hi = 126;                  // largest code lo with value(lo) * gd <= num
  while (lo < hi) {
    const uint32_t mid = (lo + hi + 1) >> 1;
    if (e4m3_f64(mid) * gd <= num) lo = mid;
    else hi = mid - 1;
  }
  if (lo == 126) return 126;
  const double twice_mid = (e4m3_f64(lo) + e4m3_f64(lo + 1)) * gd;
  const double twice_num = 2.0 * num;
  if (twice_num > twice_mid) return lo + 1;
  if (twice_num < twice_mid) return lo;
  return (lo & 1u) ? lo + 1 : lo;
}

__global__ __launch_bounds__(kPackThreads) void harmonize_kernel(uint8_t* __restrict__ packed, uint32_t N,
                                                                uint32_t kb_valid, uint32_t kc_count,
                                                                uint32_t scale_offset, SegTable segs,
                                                                const float* __restrict__ g_seg,
                                                                float* __restrict__ g_shared) {
  float gsh = 0.0f;
  for (int s = 0; s < segs.n_seg; ++s) {
    const float g = g_seg[s];
    if (g > 0.0f && (gsh == 0.0f || g < gsh)) gsh = g;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *g_shared = gsh;
  const uint32_t n_blocks = N * kb_valid;
  for (uint32_t b = blockIdx.x * kPackThreads + threadIdx.x; b < n_blocks; b += gridDim.x * kPackThreads) {
    const uint32_t n = b / kb_valid, kb = b - n * kb_valid;
    const float g = g_seg[segment_of(segs, n)];
    if (g == 0.0f || g == gsh) continue;     // all-zero segment, or ratio 1
    uint8_t* sp = packed + scale_offset + packed_scale_offset(n, kb, kc_count);
    *sp = (uint8_t)fold_scale_code(*sp, (double)gsh, (double)g);
  }
}

static SegTable make_segs(const int64_t* seg_offsets, int n_seg) {
  SegTable t{};
  t.n_seg = n_seg;
  for (int i = 0; i <= n_seg; ++i) t.off[i] = (uint32_t)seg_offsets[i];
  for (int i = n_seg + 1; i < 9; ++i) t.off[i] = t.off[n_seg];
  return t;
}

static int grid_cap(uint64_t items, int cap) {
  uint64_t g = (items + kPackThreads - 1) / kPackThreads;
  return g < 1 ? 1 : (g > (uint64_t)cap ? cap : (int)g);
}

hipError_t launch_pack_weight(const void* w, int64_t N, int64_t K, int64_t ldw,
                              const int64_t* seg_offsets, int n_seg, float* g_enc_seg,
                              bool dynamic, void* packed, float* partial, hipStream_t stream) {
  const uint16_t* wp = static_cast<const uint16_t*>(w);
  SegTable segs = make_segs(seg_offsets, n_seg);
  PackedDims d = packed_dims(N, K);
  if (dynamic) {
    hipLaunchKernelGGL(seg_amax_kernel, dim3(kWeightPartials, n_seg), dim3(kPackThreads), 0, stream,
                       wp, (uint32_t)(K / 8), (uint32_t)ldw, segs, partial);
    hipLaunchKernelGGL(seg_finalize_kernel, dim3(1), dim3(kPackThreads), 0, stream,
                       (const float*)partial, kWeightPartials, n_seg, g_enc_seg);
  }
  const uint32_t kb_pad = (uint32_t)(d.kp / 16);
  const uint32_t n_blocks_pad = (uint32_t)(d.np * kb_pad);
  hipLaunchKernelGGL(pack_kernel, dim3(grid_cap(n_blocks_pad, 8192)), dim3(kPackThreads), 0, stream,
                     wp, (uint32_t)N, (uint32_t)(K / 16), (uint32_t)ldw, kb_pad, n_blocks_pad,
                     (uint32_t)d.kc, segs, (const float*)g_enc_seg,
                     static_cast<uint8_t*>(packed), (uint32_t)d.scale_offset);
  return hipGetLastError();
}

hipError_t launch_harmonize_weight(void* packed, int64_t N, int64_t K, const int64_t* seg_offsets,
                                   int n_seg, const float* g_enc_seg, float* g_shared,
                                   hipStream_t stream) {
  SegTable segs = make_segs(seg_offsets, n_seg);
  PackedDims d = packed_dims(N, K);
  const uint32_t kb_valid = (uint32_t)(K / 16);
  hipLaunchKernelGGL(harmonize_kernel, dim3(grid_cap((uint64_t)N * kb_valid, 4096)), dim3(kPackThreads), 0,
                     stream, static_cast<uint8_t*>(packed), (uint32_t)N, kb_valid, (uint32_t)d.kc,
                     (uint32_t)d.scale_offset, segs, g_enc_seg, g_shared);
  return hipGetLastError();
}

hipError_t launch_unpack_weight(const void* packed, int64_t N, int64_t K, uint8_t* codes,
                                uint8_t* scales, hipStream_t stream) {
  PackedDims d = packed_dims(N, K);
  const uint32_t kb_valid = (uint32_t)(K / 16);
  hipLaunchKernelGGL(unpack_kernel, dim3(grid_cap((uint64_t)N * kb_valid, 8192)), dim3(kPackThreads), 0,
                     stream, static_cast<const uint8_t*>(packed), (uint32_t)N, kb_valid, (uint32_t)d.kc,
                     (uint32_t)d.scale_offset, codes, scales);
  return hipGetLastError();
}

}  // namespace nvfp4
