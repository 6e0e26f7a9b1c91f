// NVFP4 x NVFP4 GEMM with FP32 accumulation and a per-segment scaled
// epilogue, for gfx950 (paper, section 2: W4A4 GEMM on 4-bit operands;
// section 6: each fused segment scaled by its own module's global scale).
//
// Operand path.  CDNA4 has no MFMA that takes E4M3 scales per 16 elements
// (its block-scaled MFMAs take power-of-two scales per 32), so both operands
// are decoded exactly to FP16: an E2M1 value times an E4M3 scale has at most
// 6 significant bits and lies in [2^-10, 2688], inside FP16's normal range.
// The products of two decoded values are exact in FP32 and the MFMA
// accumulates in FP32; the global scales are applied once in the epilogue.
//
// Decode: v_cvt_scalef32_pk_f16_fp4 turns 2 packed codes into 2 FP16 values
// (its scale operand only contributes a power of two, so it is left at 1.0)
// and v_pk_mul_f16 multiplies the pair by the E4M3 block scale (converted
// from its code with v_cvt_f32_fp8).  Lane l = 32 h + r of a wave supplies
// row r of a 32-row fragment and 8 consecutive reduction indices, which is
// exactly 4 bytes of packed codes under one block scale; see packed_layout.h
// for the index map shared by the activation and the prepacked weight.
//
// Tiling.  A workgroup of WM x WN waves computes a (WM*FM*32) x (WN*FN*32)
// tile; each wave owns FM x FN accumulator fragments of 32 x 32 and decodes
// its own FM + FN operand fragments per 16-deep step.  Operands are loaded
// straight from global memory (L2) into registers with raw buffer loads,
// one 64-deep chunk ahead of the MFMAs; out-of-range rows are clamped and the
// buffer bounds return zeros past the end of each tensor.  Workgroups are
// remapped so that each XCD (its own L2) runs a contiguous, M-grouped range
// of tiles.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.h"
#include "packed_layout.h"

namespace nvfp4 {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef int int4v __attribute__((ext_vector_type(4)));

constexpr int kNumXcd = 8;
constexpr int kGroupM = 8;

struct GemmParams {
  uint32_t M, N, K, ldy;
  uint32_t chunks;          // ceil(K / 64) chunks in the K loop
  uint32_t w_kc, w_kg;      // packed-weight chunk and group counts
  uint32_t w_scale_offset;  // byte offset of the packed scale region
  uint32_t w_tiles;         // Np / 32
  uint32_t a_code_bytes, a_scale_bytes, w_bytes;
  uint32_t tiles_m, tiles_n;
  int n_seg;
  uint32_t seg_off[NVFP4_SEG_TABLE];
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// E4M3 scale byte `sel` of a dword -> (S, S) in FP16 (exact: 4 significant
// bits, 2^-9 <= S <= 448).
template <int kSel>
__device__ __forceinline__ half2v scale_pair(uint32_t bytes) {
  float s = __builtin_amdgcn_cvt_f32_fp8((int)bytes, kSel);
  return __builtin_bit_cast(half2v, __builtin_amdgcn_cvt_pkrtz(s, s));
}

// 8 packed E2M1 codes (one dword) times a block scale -> 8 FP16 values in
// MFMA operand order (byte j holds elements 2j (low nibble) and 2j+1).
__device__ __forceinline__ half8 decode8(uint32_t c, half2v s) {
  half2v p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 0) * s;
  half2v p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 1) * s;
  half2v p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 2) * s;
  half2v p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(c, 1.0f, 3) * s;
  return half8{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);     // finite inputs
  return (uint16_t)(u >> 16);
}

// One 64-deep chunk of operands for a wave: FM activation fragments and FN
// weight fragments, 16 code bytes and 2 scale bytes each per lane.
template <int FM, int FN>
struct Chunk {
  int4v a[FM];
  int4v b[FN];
  uint32_t sa[FM];   // low 2 bytes: scales of blocks 4 kc + 2h + {0, 1}
  uint32_t sb[FN];
};

template <int FM, int FN, bool kAlignedK>
__device__ __forceinline__ void load_chunk(Chunk<FM, FN>& ch, uint32_t kc, const GemmParams& p,
                                           __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rs,
                                           __amdgpu_buffer_rsrc_t rw, const uint32_t (&a_row)[FM],
                                           const uint32_t (&b_tile)[FN], uint32_t lane) {
  const uint32_t h = lane >> 5;
  const uint32_t kbq = p.K >> 4;                         // blocks per row
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    ch.a[f] = __builtin_amdgcn_raw_buffer_load_b128(ra, a_row[f] * (p.K >> 1) + kc * 32u + h * 16u, 0, 0);
    const uint32_t blk = kc * 4u + 2u * h;
    const uint32_t soff = a_row[f] * kbq + blk;
    if (kAlignedK) {
      ch.sa[f] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rs, soff, 0, 0);
    } else {
      uint32_t s0 = blk < kbq ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(rs, soff, 0, 0) : 0u;
      uint32_t s1 = blk + 1 < kbq ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(rs, soff + 1, 0, 0) : 0u;
      ch.sa[f] = (s0 & 0xFFu) | ((s1 & 0xFFu) << 8);
    }
  }
#pragma unroll
  for (int f = 0; f < FN; ++f) {
    ch.b[f] = __builtin_amdgcn_raw_buffer_load_b128(rw, (b_tile[f] * p.w_kc + kc) * 1024u + lane * 16u, 0, 0);
    const uint32_t soff = p.w_scale_offset + ((b_tile[f] * p.w_kg + (kc >> 2)) * 64u + lane) * 8u + (kc & 3u) * 2u;
    ch.sb[f] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rw, soff, 0, 0);
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
__global__ __launch_bounds__(WM * WN * 64) void gemm_kernel(const uint8_t* __restrict__ a_codes,
                                                           const uint8_t* __restrict__ a_scales,
                                                           const float* __restrict__ a_g,
                                                           const uint8_t* __restrict__ w_packed,
                                                           const float* __restrict__ w_g,
                                                           void* __restrict__ y, GemmParams p) {
  constexpr int BM = WM * FM * 32, BN = WN * FN * 32;
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t r = lane & 31, h = lane >> 5;

  // Tile index: XCD-contiguous remap, then M-grouped order.
  const uint32_t total = p.tiles_m * p.tiles_n;
  const uint32_t pid0 = blockIdx.x;
  const uint32_t xcd = pid0 % kNumXcd, per = total / kNumXcd, extra = total % kNumXcd;
  const uint32_t pid = xcd * per + (xcd < extra ? xcd : extra) + pid0 / kNumXcd;
  const uint32_t in_group = kGroupM * p.tiles_n;
  const uint32_t first_m = (pid / in_group) * kGroupM;
  const uint32_t gm = (p.tiles_m - first_m) < (uint32_t)kGroupM ? (p.tiles_m - first_m) : (uint32_t)kGroupM;
  const uint32_t tm = first_m + (pid % in_group) % gm;
  const uint32_t tn = (pid % in_group) / gm;

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

  // Epilogue: y = acc / (G_A * G_W[s]) for the segment s of each column.
  const float ga = *a_g;
#pragma unroll
  for (int fb = 0; fb < FN; ++fb) {
    const uint32_t col = n0 + fb * 32 + r;
    int s = 0;
#pragma unroll
    for (int i = 1; i < NVFP4_SEG_TABLE - 1; ++i) s += (i < p.n_seg && col >= p.seg_off[i]) ? 1 : 0;
    const float prod = ga * w_g[s];
    const float alpha = prod == 0.0f ? 0.0f : 1.0f / prod;
#pragma unroll
    for (int fa = 0; fa < FM; ++fa) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t row = m0 + fa * 32 + (i >> 2) * 8 + h * 4 + (i & 3);
        if (row < p.M && col < p.N) {
          const float v = acc[fa][fb][i] * alpha;
          if (kF32Out)
            static_cast<float*>(y)[(size_t)row * p.ldy + col] = v;
          else
            static_cast<uint16_t*>(y)[(size_t)row * p.ldy + col] = f32_to_bf16_rne(v);
        }
      }
    }
  }
}

template <int WM, int WN, int FM, int FN>
static hipError_t launch_cfg(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                             const void* w_packed, const float* w_g, void* y, GemmParams p,
                             bool out_f32, bool aligned, hipStream_t stream) {
  constexpr int BM = WM * FM * 32, BN = WN * FN * 32;
  p.tiles_m = (p.M + BM - 1) / BM;
  p.tiles_n = (p.N + BN - 1) / BN;
  const dim3 grid(p.tiles_m * p.tiles_n), block(WM * WN * 64);
  const uint8_t* wp = static_cast<const uint8_t*>(w_packed);
#define NVFP4_G(F32, AL)                                                                          \
  hipLaunchKernelGGL((gemm_kernel<WM, WN, FM, FN, F32, AL>), grid, block, 0, stream, a_codes, a_scales, \
                     a_g, wp, w_g, y, p)
  if (out_f32) {
    if (aligned) NVFP4_G(true, true); else NVFP4_G(true, false);
  } else {
    if (aligned) NVFP4_G(false, true); else NVFP4_G(false, false);
  }
#undef NVFP4_G
  return hipGetLastError();
}

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                       int64_t M, int64_t K, const void* w_packed, int64_t N,
                       const int64_t* seg_offsets, int n_seg, const float* w_g, void* y,
                       int64_t ldy, bool out_f32, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  PackedDims d = packed_dims(N, K);
  GemmParams p{};
  p.M = (uint32_t)M;
  p.N = (uint32_t)N;
  p.K = (uint32_t)K;
  p.ldy = (uint32_t)ldy;
  p.chunks = (uint32_t)((K + 63) / 64);
  p.w_kc = (uint32_t)d.kc;
  p.w_kg = (uint32_t)d.kg;
  p.w_scale_offset = (uint32_t)d.scale_offset;
  p.w_tiles = (uint32_t)(d.np / 32);
  p.a_code_bytes = (uint32_t)(M * K / 2);
  p.a_scale_bytes = (uint32_t)(M * K / 16);
  p.w_bytes = (uint32_t)d.bytes;
  p.n_seg = n_seg;
  for (int i = 0; i < NVFP4_SEG_TABLE; ++i)
    p.seg_off[i] = (uint32_t)seg_offsets[i <= n_seg ? i : n_seg];
  const bool aligned = (K % 64) == 0;
  if (N <= 96)
    return launch_cfg<4, 1, 2, 3>(a_codes, a_scales, a_g, w_packed, w_g, y, p, out_f32, aligned, stream);
  return launch_cfg<2, 2, 4, 4>(a_codes, a_scales, a_g, w_packed, w_g, y, p, out_f32, aligned, stream);
}

}  // namespace nvfp4
