// Register-path NVFP4 GEMM (K % 64 != 0): operands go global -> registers
// one chunk ahead; per-block masking of the scales handles a K tail.
#include "gemm_common.h"

namespace nvfp4 {

// One 64-deep chunk of operands for a wave: FM activation fragments and FN
// weight fragments, 16 code bytes and 2 scale bytes each per lane.
template <int FM, int FN>
struct Chunk {
  int4v a[FM];
  int4v b[FN];
  // Scales of blocks 4 kc + 2h + {0, 1} (bytes 0 and 1).  Kept as loaded:
  // any widening is left to the consumer, so that no instruction right after
  // the loads waits for them.
  uint16_t sa[FM];
  uint16_t sb[FN];
};

template <int FM, int FN, bool kAlignedK>
__device__ __forceinline__ void load_chunk(Chunk<FM, FN>& ch, uint32_t kc, const GemmParams& p,
                                           __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rs,
                                           __amdgpu_buffer_rsrc_t rw, const uint32_t (&a_row)[FM],
                                           const uint32_t (&b_tile)[FN], uint32_t lane) {
  const uint32_t h = lane >> 5, r = lane & 31;
  const uint32_t kbq = p.K >> 4;                         // blocks per row
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    ch.a[f] = __builtin_amdgcn_raw_buffer_load_b128(ra, a_row[f] * (p.K >> 1) + kc * 32u + h * 16u, 0, 0);
    const uint32_t blk = kc * 4u + 2u * h;
    const uint32_t soff = a_row[f] * kbq + blk;
    if (kAlignedK) {
      ch.sa[f] = __builtin_amdgcn_raw_buffer_load_b16(rs, soff, 0, 0);
    } else {
      uint32_t s0 = blk < kbq ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(rs, soff, 0, 0) : 0u;
      uint32_t s1 = blk + 1 < kbq ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(rs, soff + 1, 0, 0) : 0u;
      ch.sa[f] = (uint16_t)((s0 & 0xFFu) | ((s1 & 0xFFu) << 8));
    }
  }
#pragma unroll
  for (int f = 0; f < FN; ++f) {
    ch.b[f] = __builtin_amdgcn_raw_buffer_load_b128(rw, (b_tile[f] * p.w_kc + kc) * 1024u + lane * 16u, 0, 0);
    const uint32_t soff = p.w_scale_offset + ((b_tile[f] * p.w_kc + kc) * 32u + r) * 4u + 2u * h;
    ch.sb[f] = __builtin_amdgcn_raw_buffer_load_b16(rw, soff, 0, 0);
  }
}

template <int FM, int FN>
__device__ __forceinline__ void mma_chunk(floatx16 (&acc)[FM][FN], const Chunk<FM, FN>& ch) {
  half2v sa[FM][2], sb[FN][2];
#pragma unroll
  for (int f = 0; f < FM; ++f) { sa[f][0] = scale_pair<0>(ch.sa[f]); sa[f][1] = scale_pair<1>(ch.sa[f]); }
#pragma unroll
  for (int f = 0; f < FN; ++f) { sb[f][0] = scale_pair<0>(ch.sb[f]); sb[f][1] = scale_pair<1>(ch.sb[f]); }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    half8 av[FM], bv[FN];
#pragma unroll
    for (int f = 0; f < FM; ++f) av[f] = decode8((uint32_t)ch.a[f][j], sa[f][j >> 1]);
#pragma unroll
    for (int f = 0; f < FN; ++f) bv[f] = decode8((uint32_t)ch.b[f][j], sb[f][j >> 1]);
#pragma unroll
    for (int fa = 0; fa < FM; ++fa)
#pragma unroll
      for (int fb = 0; fb < FN; ++fb)
        acc[fa][fb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[fa], bv[fb], acc[fa][fb], 0, 0, 0);
  }
}

template <int WM, int WN, int FM, int FN, bool kF32Out, bool kAlignedK>
__global__ __launch_bounds__(WM * WN * 64) void gemm_reg_kernel(const uint8_t* __restrict__ a_codes,
                                                               const uint8_t* __restrict__ a_scales,
                                                               const float* __restrict__ a_g,
                                                               const uint8_t* __restrict__ w_packed,
                                                               const float* __restrict__ w_g,
                                                               void* __restrict__ y, GemmParams p) {
  constexpr int BM = WM * FM * 32, BN = WN * FN * 32;
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t r = lane & 31, h = lane >> 5;
  uint32_t tm, tn;
  tile_of<8>(p, tm, tn);
  const uint32_t wm = wave / WN, wn = wave % WN;
  const uint32_t m0 = tm * BM + wm * FM * 32, n0 = tn * BN + wn * FN * 32;

  uint32_t a_row[FM], b_tile[FN];
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    uint32_t row = m0 + f * 32 + r;
    a_row[f] = row < p.M ? row : p.M - 1;
  }
#pragma unroll
  for (int f = 0; f < FN; ++f) {
    uint32_t t = (n0 >> 5) + f;
    b_tile[f] = t < p.w_tiles ? t : p.w_tiles - 1;
  }

  const __amdgpu_buffer_rsrc_t ra = rsrc(a_codes, p.a_code_bytes);
  const __amdgpu_buffer_rsrc_t rs = rsrc(a_scales, p.a_scale_bytes);
  const __amdgpu_buffer_rsrc_t rw = rsrc(w_packed, p.w_bytes);

  floatx16 acc[FM][FN];
#pragma unroll
  for (int fa = 0; fa < FM; ++fa)
#pragma unroll
    for (int fb = 0; fb < FN; ++fb) acc[fa][fb] = floatx16{};

  Chunk<FM, FN> cur, nxt;
  load_chunk<FM, FN, kAlignedK>(cur, 0, p, ra, rs, rw, a_row, b_tile, lane);
  for (uint32_t kc = 0; kc + 1 < p.chunks; ++kc) {
    load_chunk<FM, FN, kAlignedK>(nxt, kc + 1, p, ra, rs, rw, a_row, b_tile, lane);
    mma_chunk<FM, FN>(acc, cur);
    cur = nxt;
  }
  mma_chunk<FM, FN>(acc, cur);
  store_tile<FM, FN, kF32Out>(acc, p, a_g, w_g, y, m0, n0, r, h);
}

template <int WM, int WN, int FM, int FN>
static hipError_t launch_reg(const GemmOperands& o, GemmParams p, bool out_f32, bool aligned, hipStream_t stream) {
  constexpr int BM = WM * FM * 32, BN = WN * FN * 32;
  p.tiles_m = (p.M + BM - 1) / BM;
  p.tiles_n = (p.N + BN - 1) / BN;
  const dim3 grid(p.tiles_m * p.tiles_n), block(WM * WN * 64);
#define NVFP4_G(F32, AL)                                                                              \
  hipLaunchKernelGGL((gemm_reg_kernel<WM, WN, FM, FN, F32, AL>), grid, block, 0, stream, o.a_codes, o.a_scales, \
                     o.a_g, o.w_packed, o.w_g, o.y, p)
  if (out_f32) {
    if (aligned) NVFP4_G(true, true); else NVFP4_G(true, false);
  } else {
    if (aligned) NVFP4_G(false, true); else NVFP4_G(false, false);
  }
#undef NVFP4_G
  return hipGetLastError();
}

hipError_t launch_reg_square(const GemmOperands& o, GemmParams p, bool out_f32, bool aligned, hipStream_t stream) {
  return launch_reg<2, 2, 4, 4>(o, p, out_f32, aligned, stream);
}

}  // namespace nvfp4
