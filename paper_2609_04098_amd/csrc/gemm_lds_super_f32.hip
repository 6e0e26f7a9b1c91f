// Prefill GEMM instantiation: LdsSquareSuper, FP32 output (see gemm_lds.h),
// and the K-halves form of the last round of tiles built on it.
#include "gemm_lds.h"

namespace nvfp4 {

hipError_t launch_lds_super_f32(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end,
                                hipStream_t stream) {
  return launch_lds_as<LdsSquareSuper, true>(o, p, n_begin, n_end, stream);
}

// Tile columns [n_begin, n_end) whose tiles would fill at most half a round
// run as twice as many workgroups, each over one half of K: segment-scaled
// FP32 partial sums into parts[2][M][halves_row(n_end - n_begin)], then
// sum_halves.
hipError_t launch_lds_super_halves(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end,
                                   float* parts, hipStream_t stream) {
  const uint32_t ldp = halves_row(n_end - n_begin);
  p.chunks /= 2;
  p.k_parts = 2;
  p.part_stride = p.M * ldp;
  p.ldy = ldp;
  GemmOperands q = o;
  // The kernel stores column c at y[row * ldy + c]: shift the base so that
  // column n_begin lands at parts[row * width].
  q.y = reinterpret_cast<void*>(reinterpret_cast<uintptr_t>(parts) - (uintptr_t)n_begin * sizeof(float));
  return launch_lds_as<LdsSquareSuper, true>(q, p, n_begin, n_end, stream);
}

// Y[row, col0 + c] = part0[row, c] + part1[row, c] for c < width (one FP32
// addition, then RNE to bf16 for bf16 output); four columns per thread
// (partial rows are halves_row(width) floats; the padding is never stored).
template <bool kF32Out>
__global__ __launch_bounds__(256) void sum_halves_kernel(const float4* __restrict__ parts, uint32_t n4, uint32_t w4,
                                                         uint32_t width, void* __restrict__ y, uint32_t ldy,
                                                         uint32_t col0) {
  for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < n4; i += gridDim.x * 256u) {
    const float4 a = parts[i], b = parts[n4 + i];
    const uint32_t row = i / w4, c = (i - row * w4) * 4u;
    const float v[4] = {a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w};
    if (kF32Out) {
      float* d = static_cast<float*>(y) + (size_t)row * ldy + col0 + c;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (c + j < width) d[j] = v[j];
    } else {
      uint16_t* d = static_cast<uint16_t*>(y) + (size_t)row * ldy + col0 + c;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (c + j < width) d[j] = f32_to_bf16_rne(v[j]);
    }
  }
}

hipError_t launch_sum_halves(const float* parts, uint32_t M, uint32_t width, void* y, uint32_t ldy, uint32_t col0,
                             bool out_f32, hipStream_t stream) {
  const uint32_t w4 = halves_row(width) / 4, n4 = M * w4;
  const uint32_t blocks = (n4 + 255) / 256;
  const dim3 grid(blocks < 2048 ? blocks : 2048), block(256);
  const float4* p4 = reinterpret_cast<const float4*>(parts);
  if (out_f32)
    hipLaunchKernelGGL(sum_halves_kernel<true>, grid, block, 0, stream, p4, n4, w4, width, y, ldy, col0);
  else
    hipLaunchKernelGGL(sum_halves_kernel<false>, grid, block, 0, stream, p4, n4, w4, width, y, ldy, col0);
  return hipGetLastError();
}

}  // namespace nvfp4
