// RMSNorm fused with NVFP4 activation quantization under a given (static)
// global scale, for gfx950.  With a calibrated activation scale (the paper
// serves its W4A4 model with scales calibrated offline, section 3
// "Checkpoints") nothing in the quantizer depends on the whole tensor, so the
// normalization of a row and the quantization of its blocks need one HBM
// pass over the activations instead of three (norm, amax, quantize).
//
//   y = RNE_bf16((x * r) * gamma),  r = 1 / sqrt(sum_k x^2 / K + eps)
//   codes, scales = the NVFP4 quantization of y (as nvfp4_quantize_act in
//                   static mode would produce from y)
//
// Rows of up to 8192 elements: two waves per row, each holding half of the
// row in registers.  Pass 1 reads the row from HBM and forms the sum of
// squares in binary32: each lane accumulates its blocks in order, two exact
// squares per v_dot2_f32_bf16, then a butterfly over the 64 lanes and the
// two waves' sums added through LDS in a fixed order.  r uses correctly
// rounded division and square root.  Pass 2 (from the registers of pass 1)
// normalizes, rounds each value to bf16 with the hardware conversion (round
// to nearest even) and quantizes 16-element blocks exactly as the
// stand-alone quantizer does.  Longer rows: one wave per row, pass 2
// re-reads the row.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "launch.h"
#include "quant_device.h"

namespace nvfp4 {

constexpr int kNormThreads = 256;          // 4 waves = 4 rows per workgroup

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, (bf16x2){(__bf16)lo, (__bf16)hi});
}

// Normalize, round to bf16 and quantize block b of one row (d0, d1: its
// 16 bf16 values).
template <bool kHuge>
__device__ __forceinline__ void norm_quant_block(uint4 d0, uint4 d1, uint32_t b, const uint4* __restrict__ gr,
                                                 float r, float g, float gd6, uint2* __restrict__ codes_row,
                                                 uint8_t* __restrict__ scales_row, uint4* __restrict__ y_row) {
  const uint4 e0 = gr[2 * b], e1 = gr[2 * b + 1];
  const uint32_t xv[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
  const uint32_t gv[8] = {e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w};
  uint32_t v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
    v[i] = pack_bf16((bf16_lo(xv[i]) * r) * bf16_lo(gv[i]), (bf16_hi(xv[i]) * r) * bf16_hi(gv[i]));
  if (y_row != nullptr) {
    y_row[2 * b] = make_uint4(v[0], v[1], v[2], v[3]);
    y_row[2 * b + 1] = make_uint4(v[4], v[5], v[6], v[7]);
  }
  uint32_t c0, c1;
  const uint32_t sc = quantize_block<kHuge>(v, g, gd6, c0, c1);
  codes_row[b] = make_uint2(c0, c1);
  scales_row[b] = (uint8_t)sc;
}

// Sum of x^2 over the lane's blocks lane, lane + 64, ... in that order, two
// squares at a time with v_dot2_f32_bf16 (each square is exact).
__device__ __forceinline__ float sumsq8(const uint32_t v[8], float acc) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const bf16x2 p = __builtin_bit_cast(bf16x2, v[i]);
    acc = __builtin_amdgcn_fdot2_f32_bf16(p, p, acc, false);
  }
  return acc;
}

// One wave per row.  kPerLane > 0: rows of at most 64 * kPerLane blocks,
// whose first-pass loads are all issued before any is used; kPerLane == 0:
// any row length (launched for rows longer than 8192 elements).  The sum is
// accumulated in the same order either way.  With kPerLane > 0 the second
// pass works on the registers of the first (X read once); otherwise it
// re-reads the row.  (Waves that walk several rows with the next row's loads
// in flight measured 12-22% slower at 8192 x 5120 than a wave per row: the
// doubled registers cut the resident waves.  A wave per row with kPerLane =
// 5 at that width: 29.8 us; two waves per row: 28.5 us.)
template <int kPerLane>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_quant_kernel(
    const uint16_t* __restrict__ x, uint32_t M, uint32_t K, uint32_t ldx, const uint16_t* __restrict__ gamma,
    float eps, const float* __restrict__ g_enc, uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    uint16_t* __restrict__ y, uint32_t ldy) {
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t row = blockIdx.x * (kNormThreads / 64) + (threadIdx.x >> 6);
  if (row >= M) return;                                     // the whole wave
  const uint32_t nb = K >> 4;
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)row * ldx);

  float ss = 0.0f;
  uint4 d[kPerLane > 0 ? kPerLane : 1][2];
  if constexpr (kPerLane > 0) {
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) {
      const uint32_t b = lane + 64u * j;
      d[j][0] = d[j][1] = make_uint4(0, 0, 0, 0);
      if (b < nb) {
        d[j][0] = xr[2 * b];
        d[j][1] = xr[2 * b + 1];
      }
    }
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) {
      const uint32_t v[8] = {d[j][0].x, d[j][0].y, d[j][0].z, d[j][0].w, d[j][1].x, d[j][1].y, d[j][1].z, d[j][1].w};
      ss = sumsq8(v, ss);
    }
  } else {
    for (uint32_t b = lane; b < nb; b += 64) {
      const uint4 d0 = xr[2 * b], d1 = xr[2 * b + 1];
      const uint32_t v[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
      ss = sumsq8(v, ss);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
  const float r = 1.0f / __builtin_sqrtf(ss / (float)K + eps);

  const float g = *g_enc;
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
  uint2* codes_row = reinterpret_cast<uint2*>(codes + (size_t)row * (K >> 1));
  uint8_t* scales_row = scales + (size_t)row * nb;
  uint4* y_row = y == nullptr ? nullptr : reinterpret_cast<uint4*>(y + (size_t)row * ldy);
  const float gd6 = g * (1.0f / 6.0f);
  auto pass2 = [&](auto huge_tag) {
    constexpr bool kHuge = decltype(huge_tag)::value;
    if constexpr (kPerLane > 0) {
      // From the registers of pass 1: X is read from memory once.
#pragma unroll
      for (int j = 0; j < kPerLane; ++j) {
        const uint32_t b = lane + 64u * j;
        if (b < nb) norm_quant_block<kHuge>(d[j][0], d[j][1], b, gr, r, g, gd6, codes_row, scales_row, y_row);
      }
    } else {
      for (uint32_t b = lane; b < nb; b += 64)
        norm_quant_block<kHuge>(xr[2 * b], xr[2 * b + 1], b, gr, r, g, gd6, codes_row, scales_row, y_row);
    }
  };
  if (g > kHugeScale)
    pass2(std::integral_constant<bool, true>{});
  else
    pass2(std::integral_constant<bool, false>{});
}

// Two waves per row (rows of at most 128 * kPerLane blocks): wave half hw
// of the row's pair takes blocks 64 hw + lane + 128 j, j < kPerLane, so each
// wave holds half of the row in registers (more resident waves than one wave
// per row); the two partial sums of squares meet in LDS and are added in the
// order half 0 + half 1.
template <int kPerLane>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_quant_pair_kernel(
    const uint16_t* __restrict__ x, uint32_t M, uint32_t K, uint32_t ldx, const uint16_t* __restrict__ gamma,
    float eps, const float* __restrict__ g_enc, uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
    uint16_t* __restrict__ y, uint32_t ldy) {
  __shared__ float half_sum[kNormThreads / 64];
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hw = wave & 1u;
  const uint32_t row = blockIdx.x * (kNormThreads / 128) + (wave >> 1);
  const bool live = row < M;                                // both waves of the pair; no early exit (barrier)
  const uint32_t nb = K >> 4;
  const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)(live ? row : 0) * ldx);
  uint4 d[kPerLane][2];
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < kPerLane; ++j) {
    const uint32_t b = 64u * hw + lane + 128u * j;
    d[j][0] = d[j][1] = make_uint4(0, 0, 0, 0);
    if (live && b < nb) {
      d[j][0] = xr[2 * b];
      d[j][1] = xr[2 * b + 1];
    }
  }
#pragma unroll
  for (int j = 0; j < kPerLane; ++j) {
    const uint32_t v[8] = {d[j][0].x, d[j][0].y, d[j][0].z, d[j][0].w, d[j][1].x, d[j][1].y, d[j][1].z, d[j][1].w};
    ss = sumsq8(v, ss);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
  if (lane == 0) half_sum[wave] = ss;
  __syncthreads();
  if (!live) return;
  ss = half_sum[wave & ~1u] + half_sum[wave | 1u];
  const float r = 1.0f / __builtin_sqrtf(ss / (float)K + eps);
  const float g = *g_enc;
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
  uint2* codes_row = reinterpret_cast<uint2*>(codes + (size_t)row * (K >> 1));
  uint8_t* scales_row = scales + (size_t)row * nb;
  uint4* y_row = y == nullptr ? nullptr : reinterpret_cast<uint4*>(y + (size_t)row * ldy);
  const float gd6 = g * (1.0f / 6.0f);
  auto pass2 = [&](auto huge_tag) {
    constexpr bool kHuge = decltype(huge_tag)::value;
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) {
      const uint32_t b = 64u * hw + lane + 128u * j;
      if (b < nb) norm_quant_block<kHuge>(d[j][0], d[j][1], b, gr, r, g, gd6, codes_row, scales_row, y_row);
    }
  };
  if (g > kHugeScale)
    pass2(std::integral_constant<bool, true>{});
  else
    pass2(std::integral_constant<bool, false>{});
}

hipError_t launch_rmsnorm_quant(const void* x, int64_t M, int64_t K, int64_t ldx, const void* gamma,
                                float eps, const float* g_enc, uint8_t* codes, uint8_t* scales, void* y,
                                int64_t ldy, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int64_t per_pair = (K / 16 + 127) / 128;
  if (per_pair <= 4) {
    const uint32_t rows_per_wg2 = kNormThreads / 128;
    const dim3 grid2((uint32_t)((M + rows_per_wg2 - 1) / rows_per_wg2));
#define NVFP4_NP(P)                                                                                          \
  hipLaunchKernelGGL(rmsnorm_quant_pair_kernel<P>, grid2, dim3(kNormThreads), 0, stream,                    \
                     static_cast<const uint16_t*>(x), (uint32_t)M, (uint32_t)K, (uint32_t)ldx,               \
                     static_cast<const uint16_t*>(gamma), eps, g_enc, codes, scales, static_cast<uint16_t*>(y), \
                     (uint32_t)ldy)
    if (per_pair <= 1) NVFP4_NP(1);
    else if (per_pair <= 2) NVFP4_NP(2);
    else if (per_pair <= 3) NVFP4_NP(3);          // K = 5120, the hidden size
    else NVFP4_NP(4);
#undef NVFP4_NP
    return hipGetLastError();
  }
  const uint32_t rows_per_wg = kNormThreads / 64;
  const dim3 grid((uint32_t)((M + rows_per_wg - 1) / rows_per_wg));
  hipLaunchKernelGGL(rmsnorm_quant_kernel<0>, grid, dim3(kNormThreads), 0, stream, static_cast<const uint16_t*>(x),
                     (uint32_t)M, (uint32_t)K, (uint32_t)ldx, static_cast<const uint16_t*>(gamma), eps, g_enc, codes,
                     scales, static_cast<uint16_t*>(y), (uint32_t)ldy);
  return hipGetLastError();
}

}  // namespace nvfp4
