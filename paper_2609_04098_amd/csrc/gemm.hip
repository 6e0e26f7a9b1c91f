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
// and v_pk_mul_f16 multiplies the pair by the E4M3 block scale.  The LDS
// kernel converts a lane's two scale codes per chunk with one
// v_cvt_scalef32_pk_f16_fp8 and selects the half with op_sel; the register
// kernel uses v_cvt_f32_fp8.  Lane l = 32 h + r of a wave supplies
// row r of a 32-row fragment and 8 consecutive reduction indices, which is
// exactly 4 bytes of packed codes under one block scale; see packed_layout.h
// for the index map shared by the activation and the prepacked weight.
//
// Three kernels:
//  * gemm_lds_kernel (K % 64 == 0, N > 96, M > 32; the prefill shapes): 256
//    threads, 256 x 256 tile, wave tile 128 x 128 (4 x 4 accumulator
//    fragments, 256 accumulator registers), one wave per SIMD; its own decode
//    VALU co-issues with its MFMAs.  Raw packed operands move global -> LDS
//    with direct-to-LDS buffer loads through a 4-stage ring (each fragment
//    loaded once per workgroup, the chunk advance in the scalar offset of
//    loop-invariant buffer descriptors); each wave reads its raw fragments of
//    the next chunk from LDS while it decodes and multiplies the current one,
//    and decodes the next chunk's first MFMA step beside the current chunk's
//    last.  One barrier per 64-deep chunk.  The loop body is a single basic
//    block in which MFMAs, decode VALU, LDS reads and the DMA issue of a
//    later chunk are interleaved (sched_group_barrier), so that the vector
//    memory queue and the VALU never stall the MFMA stream in bursts.
//  * gemm_splitk_kernel (N <= 96, the tall-skinny gate projections; M <= 32,
//    decode shapes): the output has too few 32 x 32 tiles to fill the chip,
//    so the four waves of a workgroup share one tile and split its
//    reduction, each streaming its chunks through a private LDS ring; the
//    partial sums meet in LDS.
//  * gemm_reg_kernel (K % 64 != 0, N > 96): operands go straight from global
//    memory to registers one chunk ahead; per-block masking of the scales
//    handles a K tail.
// All remap workgroups so that each XCD (its own L2) runs a contiguous,
// M-grouped range of tiles; out-of-range rows/columns read zeros through the
// buffer bounds and are not stored.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "launch.h"
#include "packed_layout.h"
#include "quant_device.h"

#define NVFP4_LDS __attribute__((address_space(3)))

namespace nvfp4 {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef int int4v __attribute__((ext_vector_type(4)));

constexpr int kNumXcd = 8;
constexpr uint32_t kOOB = 0x80000000u;     // buffer offset past every tensor: loads return 0

struct GemmParams {
  uint32_t M, N, K, ldy;
  uint32_t chunks;          // ceil(K / 64) chunks in the K loop
  uint32_t w_kc;            // packed-weight chunk count (Kp / 64)
  uint32_t w_scale_offset;  // byte offset of the packed scale region
  uint32_t w_tiles;         // Np / 32
  uint32_t a_code_bytes, a_scale_bytes, w_bytes;
  uint32_t tiles_m, tiles_n;
  uint32_t n_off;            // first output column of tile column 0 (LDS kernel; multiple of 32)
  int n_seg;
  uint32_t seg_off[NVFP4_SEG_TABLE];
  uint32_t y_pairs;          // bf16 output: y and ldy allow dword stores of column pairs
  // GDN gate epilogue (split-K kernel only): H b-columns, then H a-columns.
  const float* gate_a_log;
  const float* gate_dt_bias;
  uint32_t gate_h;
};

// The GDN gates of paper Eq. 1 from the scaled fused b|a projection v of
// column col: beta = sigmoid(b) for the first H columns; for the a-columns
// alpha = exp(-exp(A_log[h]) * softplus(a + dt_bias[h])), softplus taken as
// its argument above 20 (where log(1 + e^x) equals it to 2e-9 relative).
__device__ __forceinline__ float gdn_gate(float v, uint32_t col, const GemmParams& p) {
  if (col < p.gate_h) return 1.0f / (1.0f + expf(-v));
  const uint32_t h = col - p.gate_h;
  const float x = v + p.gate_dt_bias[h];
  const float sp = x > 20.0f ? x : log1pf(expf(x));
  return expf(-expf(p.gate_a_log[h]) * sp);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// E4M3 scale byte kSel of a dword -> (S, S) in FP16 (exact: 4 significant
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

// Direct-to-LDS buffer loads: each lane's 16 (or 4) bytes at voffset land at
// dst + 16 * lane (4 * lane); dst must be the same for the whole wave.
// The chunk advance goes in the scalar offset soffset; out-of-range per-lane
// offsets (kOOB) read zeros.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, uint8_t* dst, uint32_t voffset, uint32_t soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (NVFP4_LDS void*)dst, 16, voffset, soffset, 0, 0);
}
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t rs, uint8_t* dst, uint32_t voffset, uint32_t soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (NVFP4_LDS void*)dst, 4, voffset, soffset, 0, 0);
}

// Index of the calling wave in its workgroup, in a scalar register.
__device__ __forceinline__ uint32_t wave_index() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

// Two floats -> bf16 pair (lo, hi), round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16_rne(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, (bf16x2v){(__bf16)lo, (__bf16)hi});
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);     // finite inputs
  return (uint16_t)(u >> 16);
}

// Tile (tm, tn) of workgroup blockIdx.x: XCD-contiguous remap (workgroup i
// runs on XCD i % 8), then M-grouped order (kGroupM tiles of M per group).
template <int kGroupM>
__device__ __forceinline__ void tile_of(const GemmParams& p, uint32_t& tm, uint32_t& tn) {
  const uint32_t total = p.tiles_m * p.tiles_n;
  const uint32_t pid0 = blockIdx.x;
  const uint32_t xcd = pid0 % kNumXcd, per = total / kNumXcd, extra = total % kNumXcd;
  const uint32_t pid = xcd * per + (xcd < extra ? xcd : extra) + pid0 / kNumXcd;
  const uint32_t in_group = kGroupM * p.tiles_n;
  const uint32_t first_m = (pid / in_group) * kGroupM;
  const uint32_t gm = (p.tiles_m - first_m) < (uint32_t)kGroupM ? (p.tiles_m - first_m) : (uint32_t)kGroupM;
  tm = first_m + (pid % in_group) % gm;
  tn = (pid % in_group) / gm;
}

// Epilogue: y = acc / (G_A * G_W[s]) for the segment s of each column, BF16
// (round to nearest even) or FP32, rows/columns beyond M/N not stored.
template <int FM, int FN, bool kF32Out>
__device__ __forceinline__ void store_tile(const floatx16 (&acc)[FM][FN], const GemmParams& p,
                                           const float* __restrict__ a_g, const float* __restrict__ w_g,
                                           void* __restrict__ y, uint32_t m0, uint32_t n0, uint32_t r,
                                           uint32_t h) {
  const float ga = *a_g;
  float alpha[FN];
#pragma unroll
  for (int fb = 0; fb < FN; ++fb) {
    const uint32_t col = n0 + fb * 32 + r;
    int s = 0;
#pragma unroll
    for (int i = 1; i < NVFP4_SEG_TABLE - 1; ++i) s += (i < p.n_seg && col >= p.seg_off[i]) ? 1 : 0;
    const float prod = ga * w_g[s];
    alpha[fb] = prod == 0.0f ? 0.0f : 1.0f / prod;
  }
  if (!kF32Out && p.y_pairs && m0 + FM * 32 <= p.M && n0 + FN * 32 <= p.N) {
    // Whole fragments in range, bf16 pairs aligned: lanes r and r ^ 1 trade
    // halves so that each stores two adjacent columns of one row as one
    // dword (even lane: rows 4g + {0, 1}; odd lane: rows 4g + {2, 3}).  The
    // conversion is the hardware round to nearest even.
    const bool odd = (r & 1u) != 0;
    const uint32_t sel_a = odd ? 0x01000504u : 0x05040100u;   // low halves: (col even, col odd)
    const uint32_t sel_b = odd ? 0x03020706u : 0x07060302u;   // high halves
    const uint32_t col0 = n0 + (r & ~1u);
#pragma unroll
    for (int fa = 0; fa < FM; ++fa) {
#pragma unroll
      for (int fb = 0; fb < FN; ++fb) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const floatx16& v = acc[fa][fb];
          const uint32_t pk0 = pack_bf16_rne(v[4 * g] * alpha[fb], v[4 * g + 1] * alpha[fb]);       // rows +0, +1
          const uint32_t pk1 = pack_bf16_rne(v[4 * g + 2] * alpha[fb], v[4 * g + 3] * alpha[fb]);   // rows +2, +3
          const uint32_t own = odd ? pk1 : pk0;
          const uint32_t recv = (uint32_t)__builtin_amdgcn_mov_dpp((int)(odd ? pk0 : pk1), 0xB1, 0xF, 0xF, false);
          const uint32_t row = m0 + fa * 32 + g * 8 + h * 4 + (odd ? 2u : 0u);
          uint32_t* dst = reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(y) + (size_t)row * p.ldy + col0 + fb * 32);
          dst[0] = __builtin_amdgcn_perm(recv, own, sel_a);
          *reinterpret_cast<uint32_t*>(reinterpret_cast<uint16_t*>(dst) + p.ldy) = __builtin_amdgcn_perm(recv, own, sel_b);
        }
      }
    }
    return;
  }
#pragma unroll
  for (int fb = 0; fb < FN; ++fb) {
    const uint32_t col = n0 + fb * 32 + r;
#pragma unroll
    for (int fa = 0; fa < FM; ++fa) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint32_t row = m0 + fa * 32 + (i >> 2) * 8 + h * 4 + (i & 3);
        if (row < p.M && col < p.N) {
          const float v = acc[fa][fb][i] * alpha[fb];
          if (kF32Out)
            static_cast<float*>(y)[(size_t)row * p.ldy + col] = v;
          else
            static_cast<uint16_t*>(y)[(size_t)row * p.ldy + col] = f32_to_bf16_rne(v);
        }
      }
    }
  }
}

// ------------------------------------------------------------------ LDS path

namespace lds {
// s_waitcnt immediates (gfx9 encoding: vmcnt in bits [3:0] and [15:14],
// expcnt [6:4], lgkmcnt [11:8]; all-ones means "do not wait").
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kWaitLgkm0 = 0xC07F;                                    // lgkmcnt(0)
}  // namespace lds

// Workgroup shape of the LDS kernel: WM x WN waves, each owning an
// FM x FN block of 32 x 32 accumulator fragments; kOcc workgroups per CU.
template <int WM_, int WN_, int FM_, int FN_, int kOcc_, int kValu_, int kStages_, bool kSuper_ = false>
struct LdsCfg {
  static constexpr int WM = WM_, WN = WN_, FM = FM_, FN = FN_, kOcc = kOcc_;
  // kSuper (K % 256 == 0): the scales of 4 consecutive chunks move together,
  // one 16-byte DMA per fragment pair (a row's 4 scale dwords are
  // contiguous), into two alternating scale "super-stages" beside the ring.
  static constexpr bool kSuper = kSuper_;
  static constexpr int kWaves = WM * WN, kThreads = kWaves * 64;
  static constexpr int BM = WM * FM * 32, BN = WN * FN * 32;
  static constexpr int NFA = WM * FM, NFB = WN * FN;         // fragments per workgroup
  // Each wave moves the same number of A and B fragments (codes + scales).
  static constexpr int kAPerWave = NFA / kWaves, kBPerWave = NFB / kWaves;
  // Scales: one dword of 4 block scales per fragment row and chunk.  With an
  // even count per wave, one DMA moves the scales of two fragments (64
  // distinct rows, 128 B per fragment slot); with an odd count, one DMA per
  // fragment (both half-waves load the same 32 rows; 256 B slots).
  static constexpr bool kPairA = kAPerWave % 2 == 0, kPairB = kBPerWave % 2 == 0;
  static constexpr int kSFA = kPairA ? 128 : 256, kSFB = kPairB ? 128 : 256;
  static constexpr int kSDmaA = kPairA ? kAPerWave / 2 : kAPerWave, kSDmaB = kPairB ? kBPerWave / 2 : kBPerWave;
  // One stage of the ring: raw codes (1 KB per fragment), then the scale
  // slots, of one 64-deep chunk.
  static constexpr int kA = 0, kB = NFA * 1024, kSA = kB + NFB * 1024, kSB = kSA + NFA * kSFA;
  static constexpr int kStageBytes = kSuper ? kSA : kSB + NFB * kSFB;
  // A super-stage: per A fragment [32 rows][4 chunks][4 B] (512 B), then per
  // W fragment [4 chunks][32 rows][4 B] (512 B, the packed order).
  static constexpr int kSuperB = NFA * 512, kSuperBytes = kSuperB + NFB * 512;
  // kStages 64-deep stages in the ring; iteration c refills the stage of
  // chunk c (consumed by every wave before the barrier that opens the
  // iteration) with chunk c + kStages.
  static constexpr int kStages = kStages_;
  static constexpr int kSuperBase = kStages * kStageBytes;
  static constexpr int kLdsBytes = kSuperBase + (kSuper ? 2 * kSuperBytes : 0);
  // DMA loads per chunk and wave (without the super-stage loads).
  static constexpr int kLoadsPerWave = kAPerWave + kBPerWave + (kSuper ? 0 : kSDmaA + kSDmaB);
  static constexpr int kSuperLoads = 2;          // per 4 chunks: one A pair, one W pair
  static_assert(!kSuper || (kAPerWave == 2 && kBPerWave == 2 && kStages == 4), "super-stage layout");
  static constexpr int kGroupM = 4;
  static constexpr int kMfma = 4 * FM * FN;                   // MFMAs per chunk and wave
  static constexpr int kValuPerMfma = kValu_;                 // schedule: VALU slots after each MFMA
  static constexpr int kLdsReads = 2 * (FM + FN);             // LDS reads per chunk and wave
  static constexpr int kWaitFirst = lds::vmcnt_imm((kStages - 1) * kLoadsPerWave);   // chunk 0 landed
  static constexpr int kWaitNext = lds::vmcnt_imm((kStages - 2) * kLoadsPerWave);    // chunk c + 1 landed
  // With super-stages: at chunk c the loads issued after everything chunk
  // c + 1 needs are those of chunks c - 2 and c - 1, plus the super-stage
  // loads issued with chunk c - 2 or c - 1 when that is a multiple of 4.
  static constexpr int kWaitSuper0 = lds::vmcnt_imm(2 * kLoadsPerWave);                // c % 4 in {0, 3}
  static constexpr int kWaitSuper1 = lds::vmcnt_imm(2 * kLoadsPerWave + kSuperLoads);  // c % 4 in {1, 2}
  static_assert(kStages >= 2 && (kStages - 1) * kLoadsPerWave < 64, "ring depth");
  static_assert(NFA % kWaves == 0 && NFB % kWaves == 0 && kAPerWave > 0 && kBPerWave > 0, "load split");
  static_assert(kLdsReads <= kMfma / 2 && kLoadsPerWave <= kMfma, "schedule slots");
  static_assert(kOcc * kLdsBytes <= 160 * 1024, "LDS per CU");
};

// The launched shape: 256 x 256 workgroups of 2 x 2 waves, each wave a
// 128 x 128 block (4 x 4 fragments, 256 accumulator registers), one
// workgroup per CU.  Per chunk a wave decodes 8 fragments for 64 MFMAs
// (4 VALU per MFMA); with 4 x 2 fragments and two waves per SIMD it was
// 6 per MFMA and measured 4-10% slower on the prefill shapes, as did rings
// of 3 or 6 stages.  Its own VALU co-issues with its MFMAs.
typedef LdsCfg<2, 2, 4, 4, 1, 6, 4> LdsSquare;
// The same with scale super-stages (K % 256 == 0).
typedef LdsCfg<2, 2, 4, 4, 1, 5, 4, true> LdsSquareSuper;
// 256 x 128 workgroups of 2 x 2 waves with 4 x 2 fragments, two per CU: the
// tail of a launch whose last round of square tiles would be at most half
// full (see launch_gemm).
typedef LdsCfg<2, 2, 4, 2, 2, 5, 4> LdsTall;

template <class C, bool kF32Out>
__global__ __launch_bounds__(C::kThreads, C::kOcc) void gemm_lds_kernel(const uint8_t* __restrict__ a_codes,
                                                                   const uint8_t* __restrict__ a_scales,
                                                                   const float* __restrict__ a_g,
                                                                   const uint8_t* __restrict__ w_packed,
                                                                   const float* __restrict__ w_g,
                                                                   void* __restrict__ y, GemmParams p) {
  constexpr int WN = C::WN, FM = C::FM, FN = C::FN, BM = C::BM, BN = C::BN;
  constexpr int kA = C::kA, kB = C::kB, kSA = C::kSA, kSB = C::kSB, kStages = C::kStages;
  constexpr int kStageBytes = C::kStageBytes, kAPerWave = C::kAPerWave, kBPerWave = C::kBPerWave;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const uint32_t lane = threadIdx.x & 63, wave = wave_index();
  const uint32_t r = lane & 31, h = lane >> 5;
  uint32_t tm, tn;
  tile_of<C::kGroupM>(p, tm, tn);
  const uint32_t wm = wave / WN, wn = wave % WN;

  // Per-lane offsets are fixed; the chunk advances the descriptors' base
  // (and shrinks their size) in scalar registers.  Rows >= M and tiles past
  // the packed weight get offsets beyond every descriptor: zeros.
  // Scale DMA j: lane (h, r) loads the scale dword of row r of fragment
  // j * 2 + h of the wave's pair (paired), or of fragment j (single).
  uint32_t a_off[kAPerWave], as_off[C::kSDmaA], b_off[kBPerWave], bs_off[C::kSDmaB];
  const uint32_t fa0 = kAPerWave * wave, fb0 = kBPerWave * wave;   // first fragment this wave loads
  const uint32_t nt0 = (p.n_off >> 5) + tn * (BN / 32);             // first weight tile of the tile
#pragma unroll
  for (int i = 0; i < kAPerWave; ++i) {
    const uint32_t row = tm * BM + (fa0 + i) * 32 + r;
    a_off[i] = row < p.M ? row * (p.K >> 1) + h * 16u : kOOB;
  }
#pragma unroll
  for (int j = 0; j < C::kSDmaA; ++j) {
    const uint32_t row = tm * BM + (fa0 + (C::kPairA ? 2 * j + h : j)) * 32 + r;
    as_off[j] = row < p.M ? row * (p.K >> 4) : kOOB;
  }
#pragma unroll
  for (int i = 0; i < kBPerWave; ++i) {
    const uint32_t nt = nt0 + fb0 + i;
    b_off[i] = nt < p.w_tiles ? nt * p.w_kc * 1024u + lane * 16u : kOOB;
  }
#pragma unroll
  for (int j = 0; j < C::kSDmaB; ++j) {
    const uint32_t nt = nt0 + fb0 + (C::kPairB ? 2 * j + h : j);
    bs_off[j] = nt < p.w_tiles ? nt * p.w_kc * 128u + r * 4u : kOOB;
  }
  const uint8_t* w_scales = w_packed + p.w_scale_offset;
  const uint32_t w_scale_bytes = p.w_bytes - p.w_scale_offset;

  const __amdgpu_buffer_rsrc_t ra = rsrc(a_codes, p.a_code_bytes);
  const __amdgpu_buffer_rsrc_t rs = rsrc(a_scales, p.a_scale_bytes);
  const __amdgpu_buffer_rsrc_t rb = rsrc(w_packed, p.w_scale_offset);
  const __amdgpu_buffer_rsrc_t rbs = rsrc(w_scales, w_scale_bytes);
  // DMA of chunk kc into stage kc % kStages.  The ring runs kStages - 1
  // chunks past the end of K; those stages are never read, and re-load the
  // last chunk so that every address stays inside its tensor.
  auto issue = [&](uint32_t kc) {
    uint8_t* st = smem + (kc % kStages) * kStageBytes;
    const uint32_t kq = kc < p.chunks ? kc : p.chunks - 1;
#pragma unroll
    for (int i = 0; i < kAPerWave; ++i) dma16(ra, st + kA + (fa0 + i) * 1024, a_off[i], kq * 32u);
    if constexpr (!C::kSuper) {
#pragma unroll
      for (int j = 0; j < C::kSDmaA; ++j)
        dma4(rs, st + kSA + (fa0 + (C::kPairA ? 2 * j : j)) * C::kSFA, as_off[j], kq * 4u);
    }
#pragma unroll
    for (int i = 0; i < kBPerWave; ++i) dma16(rb, st + kB + (fb0 + i) * 1024, b_off[i], kq * 1024u);
    if constexpr (!C::kSuper) {
#pragma unroll
      for (int j = 0; j < C::kSDmaB; ++j)
        dma4(rbs, st + kSB + (fb0 + (C::kPairB ? 2 * j : j)) * C::kSFB, bs_off[j], kq * 128u);
    }
  };
  // Super-stage sg (the scales of chunks 4 sg .. 4 sg + 3) into buffer
  // sg % 2: lane (h, r) loads row r of the wave's A fragment fa0 + h (16
  // bytes: 4 chunks of one row) and 16 bytes (rows 4 (r % 8) .., chunk r / 8)
  // of the 512-byte group of weight tile fb0 + h.  Groups past the end of K
  // re-load the last one.
  const uint32_t a_sup_off = [&]() {
    const uint32_t row = tm * BM + (fa0 + h) * 32 + r;
    return row < p.M ? row * (p.K >> 4) : kOOB;
  }();
  const uint32_t b_sup_off = [&]() {
    const uint32_t nt = nt0 + fb0 + h;
    return nt < p.w_tiles ? nt * p.w_kc * 128u + r * 16u : kOOB;
  }();
  auto issue_super = [&](uint32_t sg) {
    uint8_t* sb = smem + C::kSuperBase + (sg & 1u) * C::kSuperBytes;
    const uint32_t last = (p.chunks >> 2) - 1;
    const uint32_t sq = sg < last ? sg : last;
    dma16(rs, sb + fa0 * 512, a_sup_off, sq * 16u);
    dma16(rbs, sb + C::kSuperB + fb0 * 512, b_sup_off, sq * 512u);
  };

  struct Regs {
    int4v ca[FM], cb[FN];
    uint32_t sa[FM], sb[FN];   // low 16 bits: the lane's two block scales
  };
  // Lane (h, r) takes the half h of row r's scale dword (blocks 2h, 2h + 1
  // of the chunk).
  auto read_stage = [&](Regs& R, uint32_t kc) {
    const uint8_t* st = smem + (kc % kStages) * kStageBytes;
    const uint8_t* sb = smem + C::kSuperBase + ((kc >> 2) & 1u) * C::kSuperBytes;
    const uint32_t j = kc & 3u;
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      R.ca[f] = *(const int4v*)(st + kA + (wm * FM + f) * 1024 + lane * 16);
      if constexpr (C::kSuper)
        R.sa[f] = *(const uint16_t*)(sb + (wm * FM + f) * 512 + r * 16 + j * 4 + h * 2);
      else
        R.sa[f] = *(const uint16_t*)(st + kSA + (wm * FM + f) * C::kSFA + r * 4 + h * 2);
    }
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      R.cb[f] = *(const int4v*)(st + kB + (wn * FN + f) * 1024 + lane * 16);
      if constexpr (C::kSuper)
        R.sb[f] = *(const uint16_t*)(sb + C::kSuperB + (wn * FN + f) * 512 + j * 128 + r * 4 + h * 2);
      else
        R.sb[f] = *(const uint16_t*)(st + kSB + (wn * FN + f) * C::kSFB + r * 4 + h * 2);
    }
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx16{};

  // The decode of MFMA step 0 of chunk c + 1 runs beside the MFMAs of step 3
  // of chunk c, so no iteration starts with a run of VALU work in front of
  // its first MFMA (one wave per SIMD: nothing else would cover it).
  half2v sA[FM], sB[FN];
  half8 av[2][FM], bv[2][FN];
  auto scales = [&](const Regs& R) {
#pragma unroll
    for (int f = 0; f < FM; ++f) sA[f] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(R.sa[f], 1.0f, false);
#pragma unroll
    for (int f = 0; f < FN; ++f) sB[f] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(R.sb[f], 1.0f, false);
  };
  // Decode MFMA step j (0..3) of R into buffer u; steps 0, 1 use the first
  // block scale of the lane, steps 2, 3 the second.
  auto decode_step = [&](const Regs& R, int j, int u) {
#pragma unroll
    for (int f = 0; f < FM; ++f)
      av[u][f] = decode8((uint32_t)R.ca[f][j], j >> 1 ? __builtin_shufflevector(sA[f], sA[f], 1, 1)
                                                      : __builtin_shufflevector(sA[f], sA[f], 0, 0));
#pragma unroll
    for (int f = 0; f < FN; ++f)
      bv[u][f] = decode8((uint32_t)R.cb[f][j], j >> 1 ? __builtin_shufflevector(sB[f], sB[f], 1, 1)
                                                      : __builtin_shufflevector(sB[f], sB[f], 0, 0));
  };
  // One chunk: wait until chunk c + 1 has landed, barrier, DMA of chunk
  // c + kStages into the stage of chunk c (and, with super-stages, at
  // c % 4 == 0 the scales of chunks c + 4 .. c + 7 into the buffer that held
  // those of chunks c - 4 .. c - 1), LDS reads of chunk c + 1 into `next`,
  // decode + MFMA of `cur`.  pos_tag: c % 4 (super-stages) or 0.
  auto step = [&](uint32_t c, const Regs& cur, Regs& next, auto pos_tag) {
    constexpr int kPos = decltype(pos_tag)::value;
    constexpr bool kIssueSuper = C::kSuper && kPos == 0;
    // Every LDS read of the previous iteration has been consumed by its
    // decode, so after the barrier the stage of chunk c may be refilled.
    if constexpr (C::kSuper)
      __builtin_amdgcn_s_waitcnt(kPos == 1 || kPos == 2 ? C::kWaitSuper1 : C::kWaitSuper0);
    else
      __builtin_amdgcn_s_waitcnt(C::kWaitNext);
    __builtin_amdgcn_s_barrier();
    issue(c + kStages);
    if constexpr (kIssueSuper) issue_super((c >> 2) + 1);
    read_stage(next, c + 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int u = j & 1;
      if (j < 3) {
        decode_step(cur, j + 1, u ^ 1);
      } else {
        scales(next);
        decode_step(next, 0, 0);
      }
#pragma unroll
      for (int fa = 0; fa < FM; ++fa)
#pragma unroll
        for (int fb = 0; fb < FN; ++fb)
          acc[fa][fb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[u][fa], bv[u][fb], acc[fa][fb], 0, 0, 0);
    }
    // LDS reads spread over the first half of the chunk, DMA issues over the
    // first three quarters.
    constexpr int kDma = C::kLoadsPerWave + (kIssueSuper ? C::kSuperLoads : 0);
    constexpr int kLdsEvery = (C::kMfma / 2) / C::kLdsReads;
    constexpr int kDmaEvery = (3 * C::kMfma / 4) / kDma;
#pragma unroll
    for (int i = 0; i < C::kMfma; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                       // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, C::kValuPerMfma, 0);         // VALU
      if (i % kLdsEvery == kLdsEvery - 1 && i / kLdsEvery < C::kLdsReads)
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);                     // LDS read
      if (i % kDmaEvery == 0 && i / kDmaEvery < kDma)
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                     // VMEM (DMA)
    }
  };
  using Pos0 = std::integral_constant<int, 0>;
  using Pos1 = std::integral_constant<int, 1>;
  using Pos2 = std::integral_constant<int, 2>;
  using Pos3 = std::integral_constant<int, 3>;

  if constexpr (C::kSuper) {
    issue_super(0);                          // before chunk 0's codes: landed with them
    __builtin_amdgcn_sched_barrier(0);       // keep that order (the waits count loads in issue order)
  }
#pragma unroll
  for (int s = 0; s < kStages; ++s) issue(s);
  __builtin_amdgcn_s_waitcnt(C::kWaitFirst);
  __builtin_amdgcn_s_barrier();
  Regs cur, nxt;
  read_stage(cur, 0);
  scales(cur);
  decode_step(cur, 0, 0);
  if constexpr (C::kSuper) {
    // p.chunks % 4 == 0 (K % 256 == 0).
    for (uint32_t c = 0; c < p.chunks; c += 4) {
      step(c, cur, nxt, Pos0{});
      step(c + 1, nxt, cur, Pos1{});
      step(c + 2, cur, nxt, Pos2{});
      step(c + 3, nxt, cur, Pos3{});
    }
  } else {
    for (uint32_t c = 0; c < p.chunks; ++c) {
      step(c, cur, nxt, Pos0{});
      cur = nxt;
    }
  }
  // Drain the DMA of the chunks past the end before the workgroup exits.
  __builtin_amdgcn_s_waitcnt(0x0F70);
  store_tile<FM, FN, kF32Out>(acc, p, a_g, w_g, y, tm * BM + wm * FM * 32, p.n_off + tn * BN + wn * FN * 32, r, h);
}

// ------------------------------------------------------------- register path

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

// ----------------------------------------------------------- split-K path
//
// Shapes whose output has too few 32 x 32 tiles to give every SIMD two waves
// (N <= 96: the tall-skinny gate projections; M <= 32: decode-shaped calls,
// weight-bandwidth-bound): the KS waves of a workgroup share one FM x FN
// fragment tile and split its reduction, wave w taking chunks w, w + KS, ...
// Each wave streams its own chunks through a private LDS ring with
// direct-to-LDS loads (no barrier in the loop; its own memory counter says
// when a stage has landed), reads the next chunk's raw fragments from LDS
// while it decodes and multiplies the current one, and the partial sums meet
// in LDS at the end; fragment f is summed in wave order (deterministic) and
// stored by wave f % KS.  Requires K % 64 == 0.
// 1 / (G_A G_W[s]) for the column of lane r in each of the FN fragment
// columns of a tile (0 when either scale is 0).  Taken before the main loop,
// so that the loads of the scales are off the epilogue's path.
template <int FN>
__device__ __forceinline__ void segment_alpha(const GemmParams& p, float ga, const float* __restrict__ w_g,
                                              uint32_t n0, uint32_t r, float (&alpha)[FN]) {
#pragma unroll
  for (int fb = 0; fb < FN; ++fb) {
    const uint32_t col = n0 + fb * 32 + r;
    int s = 0;
#pragma unroll
    for (int i = 1; i < NVFP4_SEG_TABLE - 1; ++i) s += (i < p.n_seg && col >= p.seg_off[i]) ? 1 : 0;
    const float prod = ga * w_g[s];
    alpha[fb] = prod == 0.0f ? 0.0f : 1.0f / prod;
  }
}

// Split-K epilogue: the KS waves' partial sums meet in LDS, kGroup fragments
// at a time (part: kGroup x KS x 64 floatx16), and are summed in wave order
// (deterministic).  Plain outputs: fragment f is summed and stored by wave
// f % KS.  With the GDN gate transform (kGate), whose transcendentals
// dominate the epilogue, every wave takes 16 / KS of each lane's 16
// accumulator entries of every fragment instead, so that all waves share
// that arithmetic.  Each value is scaled by its column's alpha.  LDS at part
// must be free (a caller that used it for other data synchronizes first).
template <int KS, int FM, int FN, int kGroup, bool kF32Out, bool kGate>
__device__ __forceinline__ void splitk_epilogue(const floatx16 (&acc)[FM][FN], floatx16* part, const GemmParams& p,
                                                const float (&alpha)[FN], void* __restrict__ y,
                                                uint32_t m0, uint32_t n0, uint32_t wave, uint32_t lane) {
  static_assert(16 % KS == 0, "entries per wave");
  constexpr int kPer = 16 / KS, kFrags = FM * FN;
  const uint32_t r = lane & 31, h = lane >> 5;
  const float* partf = reinterpret_cast<const float*>(part);
  auto store = [&](float v, uint32_t row, uint32_t col) {
    if (row < p.M && col < p.N) {
      if (kGate) v = gdn_gate(v, col, p);
      if (kF32Out)
        static_cast<float*>(y)[(size_t)row * p.ldy + col] = v;
      else
        static_cast<uint16_t*>(y)[(size_t)row * p.ldy + col] = f32_to_bf16_rne(v);
    }
  };
#pragma unroll
  for (int g0 = 0; g0 < kFrags; g0 += kGroup) {
    if (g0 > 0) __syncthreads();                   // the previous group has been read
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
      if (g0 + j < kFrags) part[(j * KS + wave) * 64 + lane] = acc[(g0 + j) / FN][(g0 + j) % FN];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const int f = g0 + j;
      if (f >= kFrags) break;
      const int fa = f / FN, fb = f % FN;
      const uint32_t col = n0 + fb * 32 + r;
      const floatx16* pj = part + j * KS * 64;
      if (kGate) {
        const float* pf = partf + j * KS * 64 * 16;
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
          const uint32_t i = wave * kPer + e;               // accumulator entry of this wave
          float sum = pf[lane * 16 + i];
#pragma unroll
          for (int w = 1; w < KS; ++w) sum += pf[(w * 64 + lane) * 16 + i];
          store(sum * alpha[fb], m0 + fa * 32 + (i >> 2) * 8 + h * 4 + (i & 3), col);
        }
      } else if (wave == (uint32_t)(f % KS)) {
        floatx16 sum = pj[lane];
#pragma unroll
        for (int w = 1; w < KS; ++w) sum += pj[w * 64 + lane];
#pragma unroll
        for (int i = 0; i < 16; ++i) store(sum[i] * alpha[fb], m0 + fa * 32 + (i >> 2) * 8 + h * 4 + (i & 3), col);
      }
    }
  }
}

// One stage of a split-K wave's ring: FM + FN raw code fragments (1 KB
// each), then the scale dwords of the A fragments and of the W fragments,
// two fragments (256 B) per scale DMA.
template <int FM, int FN>
struct SplitkStage {
  static constexpr int kPairsA = (FM + 1) / 2, kPairsB = (FN + 1) / 2;
  static constexpr int kScaleA = (FM + FN) * 1024;
  static constexpr int kScaleB = kScaleA + kPairsA * 256;
  static constexpr int kBytes = kScaleB + kPairsB * 256;
  static constexpr int kLoads = FM + FN + kPairsA + kPairsB;
};

template <int KS, int FM, int FN, int kStages, bool kF32Out, bool kGate>
__global__ __launch_bounds__(KS * 64, 2) void gemm_splitk_kernel(const uint8_t* __restrict__ a_codes,
                                                             const uint8_t* __restrict__ a_scales,
                                                             const float* __restrict__ a_g,
                                                             const uint8_t* __restrict__ w_packed,
                                                             const float* __restrict__ w_g,
                                                             void* __restrict__ y, GemmParams p) {
  constexpr int BM = FM * 32, BN = FN * 32;
  using L = SplitkStage<FM, FN>;
  constexpr int kFrags = FM + FN;
  constexpr int kScaleA = L::kScaleA, kScaleB = L::kScaleB, kStageBytes = L::kBytes;
  constexpr int kLoads = L::kLoads;                          // DMA loads per chunk and wave
  constexpr int kWaitFirst = lds::vmcnt_imm((kStages - 1) * kLoads);
  constexpr int kWaitNext = lds::vmcnt_imm((kStages - 1) * kLoads);
  static_assert(kStages >= 2 && kStages <= 4 && (kStages - 1) * kLoads < 64, "ring depth, memory counter range");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  // The wave index is uniform: taking it through readfirstlane keeps the
  // chunk index, buffer descriptors and LDS addresses in scalar registers.
  const uint32_t lane = threadIdx.x & 63, wave = wave_index();
  const uint32_t r = lane & 31, h = lane >> 5;
  uint32_t tm, tn;
  tile_of<8>(p, tm, tn);
  const uint32_t m0 = tm * BM, n0 = tn * BN;
  uint8_t* ring = smem + wave * (kStages * kStageBytes);

  // Scale DMA of fragment pair j: lane l loads the scale dword of row l of
  // the pair (A), or of row l % 32 of weight tile l / 32 of the pair (W);
  // the missing second fragment of an odd count reads zeros.
  uint32_t a_off[FM], as_off[L::kPairsA], b_off[FN], bs_off[L::kPairsB];
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    const uint32_t row = m0 + f * 32 + r;
    a_off[f] = row < p.M ? row * (p.K >> 1) + h * 16u : kOOB;
  }
#pragma unroll
  for (int j = 0; j < L::kPairsA; ++j) {
    const uint32_t row = m0 + 2 * j * 32 + lane;
    as_off[j] = (2 * j + h < (uint32_t)FM && row < p.M) ? row * (p.K >> 4) : kOOB;
  }
#pragma unroll
  for (int f = 0; f < FN; ++f) {
    const uint32_t nt = (n0 >> 5) + f;
    b_off[f] = nt < p.w_tiles ? nt * p.w_kc * 1024u + lane * 16u : kOOB;
  }
#pragma unroll
  for (int j = 0; j < L::kPairsB; ++j) {
    const uint32_t nt = (n0 >> 5) + 2 * j + h;
    bs_off[j] = (2 * j + h < (uint32_t)FN && nt < p.w_tiles) ? nt * p.w_kc * 128u + r * 4u : kOOB;
  }
  const uint8_t* w_scales = w_packed + p.w_scale_offset;
  const uint32_t w_scale_bytes = p.w_bytes - p.w_scale_offset;
  const uint32_t n_mine = wave < p.chunks ? (p.chunks - 1 - wave) / KS + 1 : 0;
  float alpha[FN];
  segment_alpha<FN>(p, *a_g, w_g, n0, r, alpha);

  const __amdgpu_buffer_rsrc_t ra = rsrc(a_codes, p.a_code_bytes);
  const __amdgpu_buffer_rsrc_t rs = rsrc(a_scales, p.a_scale_bytes);
  const __amdgpu_buffer_rsrc_t rb = rsrc(w_packed, p.w_scale_offset);
  const __amdgpu_buffer_rsrc_t rbs = rsrc(w_scales, w_scale_bytes);
  // DMA of this wave's i-th chunk into stage i % kStages.  (Prologue loads
  // of chunks past the end of K, when K is short, re-load the last chunk so
  // that every address stays inside its tensor; they are never read.)
  auto issue = [&](uint32_t i) {
    const uint32_t kc = wave + KS * i;
    const uint32_t kq = kc < p.chunks ? kc : p.chunks - 1;
    uint8_t* st = ring + (i % kStages) * kStageBytes;
#pragma unroll
    for (int f = 0; f < FM; ++f) dma16(ra, st + f * 1024, a_off[f], kq * 32u);
#pragma unroll
    for (int j = 0; j < L::kPairsA; ++j) dma4(rs, st + kScaleA + j * 256, as_off[j], kq * 4u);
#pragma unroll
    for (int f = 0; f < FN; ++f) dma16(rb, st + (FM + f) * 1024, b_off[f], kq * 1024u);
#pragma unroll
    for (int j = 0; j < L::kPairsB; ++j) dma4(rbs, st + kScaleB + j * 256, bs_off[j], kq * 128u);
  };

  struct Regs {
    int4v c[kFrags];
    uint32_t s[kFrags];
  };
  auto read_stage = [&](Regs& R, uint32_t i) {
    const uint8_t* st = ring + (i % kStages) * kStageBytes;
#pragma unroll
    for (int f = 0; f < kFrags; ++f) {
      R.c[f] = *(const int4v*)(st + f * 1024 + lane * 16);
      R.s[f] = *(const uint32_t*)(st + (f < FM ? kScaleA + f * 128 : kScaleB + (f - FM) * 128) + r * 4);
    }
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int fa = 0; fa < FM; ++fa)
#pragma unroll
    for (int fb = 0; fb < FN; ++fb) acc[fa][fb] = floatx16{};

  // cur's stage is free once cur is in registers, so it is refilled before
  // the wait for chunk i + 1: kStages - 1 chunks stay in flight through it.
  // Near the end nothing is refilled, and the wait for chunk i + 1 lets
  // exactly the chunks after it stay in flight (loads land in order).
  auto step = [&](uint32_t i, const Regs& cur, Regs& next) {
    __builtin_amdgcn_s_waitcnt(lds::kWaitLgkm0);       // cur read from its stage
    if (i + kStages < n_mine) {
      issue(i + kStages);                               // refills cur's stage
      __builtin_amdgcn_s_waitcnt(kWaitNext);            // chunk i + 1 landed
    } else {
      const int rem = (int)n_mine - 2 - (int)i;         // chunks after i + 1 (< kStages - 1)
      if (rem >= 2)
        __builtin_amdgcn_s_waitcnt(lds::vmcnt_imm(2 * kLoads));
      else if (rem == 1)
        __builtin_amdgcn_s_waitcnt(lds::vmcnt_imm(kLoads));
      else
        __builtin_amdgcn_s_waitcnt(lds::vmcnt_imm(0));
    }
    read_stage(next, i + 1);
    half2v sc[kFrags];
#pragma unroll
    for (int f = 0; f < kFrags; ++f) sc[f] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(cur.s[f] >> (16 * h), 1.0f, false);
    half8 v[2][kFrags];
#pragma unroll
    for (int f = 0; f < kFrags; ++f) v[0][f] = decode8((uint32_t)cur.c[f][0], __builtin_shufflevector(sc[f], sc[f], 0, 0));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int u = j & 1;
      if (j < 3) {
        const int t = (j + 1) >> 1;
#pragma unroll
        for (int f = 0; f < kFrags; ++f)
          v[u ^ 1][f] = decode8((uint32_t)cur.c[f][j + 1], t ? __builtin_shufflevector(sc[f], sc[f], 1, 1)
                                                            : __builtin_shufflevector(sc[f], sc[f], 0, 0));
      }
#pragma unroll
      for (int fa = 0; fa < FM; ++fa)
#pragma unroll
        for (int fb = 0; fb < FN; ++fb)
          acc[fa][fb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(v[u][fa], v[u][FM + fb], acc[fa][fb], 0, 0, 0);
    }
    constexpr int kMfma = 4 * FM * FN;
    constexpr int kValu = (4 * 8 * kFrags + 2 * kFrags + kMfma - 1) / kMfma;
#pragma unroll
    for (int q = 0; q < kMfma; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, kValu, 0);                               // VALU
      if (q < kLoads) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                   // VMEM (DMA)
      if (q < 2 * kFrags) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);               // LDS read
    }
  };

#pragma unroll
  for (int s = 0; s < kStages; ++s) issue(s);
  __builtin_amdgcn_s_waitcnt(kWaitFirst);
  Regs cur, nxt;
  read_stage(cur, 0);
  for (uint32_t i = 0; i < n_mine; ++i) {
    step(i, cur, nxt);
    cur = nxt;
  }
  // Drain this wave's DMA (prologue loads past a short K) before the ring
  // is reused for the partial sums.
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();

  constexpr int kFit = (kStages * kStageBytes) / (64 * 64);   // fragments whose partials fit the ring
  constexpr int kGroup = kFit < FM * FN ? kFit : FM * FN;
  static_assert(kGroup >= 1, "partial sums of one fragment fit the ring");
  splitk_epilogue<KS, FM, FN, kGroup, kF32Out, kGate>(acc, reinterpret_cast<floatx16*>(smem), p, alpha, y, m0, n0,
                                                      wave, lane);
}

// ------------------------------------------- fused quantize + tall-skinny GEMM
//
// For narrow outputs (N <= 128: the gate projections), the activation is
// quantized inside the GEMM: each lane loads the 32 bf16 values it supplies
// to the MFMA (row r, reduction indices [32h, 32h + 32) of the chunk: two
// whole blocks), quantizes them with the same device code as the stand-alone
// quantizer (so the codes are identical), optionally stores the codes and
// scales, and feeds the decoded values to the MFMA; X is read once and the
// codes never travel through memory.  Tile: 32 rows x FN fragments, the KS
// waves of a workgroup split the reduction (wave w takes chunks w, w + KS,
// ...), operands go straight to registers one chunk ahead, and the partial
// sums meet in LDS (splitk_epilogue).  G_A is read (static) or formed from
// the amax pass's partial maxima (dynamic; workgroup 0 writes it out), and
// the epilogue uses the value, not the memory.  K % 64 == 0.
struct QuantGemmArgs {
  const uint16_t* x;
  uint32_t x_bytes, ldx_bytes;
  float* g_enc;
  const float* partial;
  uint32_t n_partial;
  uint8_t* codes;
  uint8_t* scales;
};

template <int KS, int FM, int FN, int kDepth, bool kDynamic, bool kF32Out, bool kCodes>
__global__ __launch_bounds__(KS * 64, 2) void quant_gemm_kernel(QuantGemmArgs q, const uint8_t* __restrict__ w_packed,
                                                            const float* __restrict__ w_g, void* __restrict__ y,
                                                            GemmParams p) {
  __shared__ floatx16 part[KS * 64];
  __shared__ uint32_t red[KS];
  const uint32_t lane = threadIdx.x & 63, wave = wave_index();
  const uint32_t r = lane & 31, h = lane >> 5;
  float g;
  if (kDynamic) {
    uint32_t m = 0;
    for (uint32_t i = threadIdx.x; i < q.n_partial; i += KS * 64) {
      const uint32_t v = __float_as_uint(q.partial[i]);
      m = m > v ? m : v;                       // non-negative floats order as integers
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const uint32_t o = __shfl_xor(m, off, 64);
      m = m > o ? m : o;
    }
    if (lane == 0) red[wave] = m;
    __syncthreads();
    m = red[0];
#pragma unroll
    for (int w = 1; w < KS; ++w) m = m > red[w] ? m : red[w];
    g = global_scale(__uint_as_float(m));
    if (blockIdx.x == 0 && threadIdx.x == 0) *q.g_enc = g;
  } else {
    g = *q.g_enc;
  }
  const float gd6 = g * (1.0f / 6.0f);
  uint32_t tm, tn;
  tile_of<8>(p, tm, tn);
  const uint32_t m0 = tm * (FM * 32), n0 = tn * (FN * 32);

  // Per-lane offsets; the chunk goes in the scalar offset.  Rows >= M read
  // zeros (an all-zero block quantizes to zero codes and is not stored).
  const __amdgpu_buffer_rsrc_t rx = rsrc(q.x, q.x_bytes);
  uint32_t x_off[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    const uint32_t row = m0 + f * 32 + r;
    x_off[f] = row < p.M ? row * q.ldx_bytes + h * 64u : kOOB;
  }
  uint32_t b_off[FN], bs_off[FN];
#pragma unroll
  for (int f = 0; f < FN; ++f) {
    const uint32_t nt = (n0 >> 5) + f;
    b_off[f] = nt < p.w_tiles ? nt * p.w_kc * 1024u + lane * 16u : kOOB;
    bs_off[f] = nt < p.w_tiles ? nt * p.w_kc * 128u + r * 4u + h * 2u : kOOB;
  }
  const __amdgpu_buffer_rsrc_t rb = rsrc(w_packed, p.w_scale_offset);
  const __amdgpu_buffer_rsrc_t rbs = rsrc(w_packed + p.w_scale_offset, p.w_bytes - p.w_scale_offset);
  const uint32_t n_mine = wave < p.chunks ? (p.chunks - 1 - wave) / KS + 1 : 0;
  float alpha[FN];
  segment_alpha<FN>(p, g, w_g, n0, r, alpha);

  struct Chunk {
    int4v x[FM][4];         // per fragment, the lane's 32 bf16 values
    int4v b[FN];
    uint32_t sb[FN];        // low 16 bits: the lane's two weight block scales
  };
  auto load = [&](Chunk& c, uint32_t i) {
    const uint32_t kc = wave + KS * i;
#pragma unroll
    for (int f = 0; f < FM; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        c.x[f][j] = __builtin_amdgcn_raw_buffer_load_b128(rx, x_off[f] + 16u * j, kc * 128u, 0);
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      c.b[f] = __builtin_amdgcn_raw_buffer_load_b128(rb, b_off[f], kc * 1024u, 0);
      c.sb[f] = __builtin_amdgcn_raw_buffer_load_b16(rbs, bs_off[f], kc * 128u, 0);
    }
  };
  floatx16 acc[FM][FN];
#pragma unroll
  for (int fa = 0; fa < FM; ++fa)
#pragma unroll
    for (int fb = 0; fb < FN; ++fb) acc[fa][fb] = floatx16{};

  auto run = [&](auto huge_tag) {
    constexpr bool kHuge = decltype(huge_tag)::value;
    auto compute = [&](const Chunk& c, uint32_t i) {
      const uint32_t kc = wave + KS * i;
      uint32_t cd[FM][4];
      half2v sa[FM];
#pragma unroll
      for (int f = 0; f < FM; ++f) {
        const uint32_t v0[8] = {(uint32_t)c.x[f][0][0], (uint32_t)c.x[f][0][1], (uint32_t)c.x[f][0][2],
                                (uint32_t)c.x[f][0][3], (uint32_t)c.x[f][1][0], (uint32_t)c.x[f][1][1],
                                (uint32_t)c.x[f][1][2], (uint32_t)c.x[f][1][3]};
        const uint32_t v1[8] = {(uint32_t)c.x[f][2][0], (uint32_t)c.x[f][2][1], (uint32_t)c.x[f][2][2],
                                (uint32_t)c.x[f][2][3], (uint32_t)c.x[f][3][0], (uint32_t)c.x[f][3][1],
                                (uint32_t)c.x[f][3][2], (uint32_t)c.x[f][3][3]};
        const uint32_t s0 = quantize_block<kHuge>(v0, g, gd6, cd[f][0], cd[f][1]);
        const uint32_t s1 = quantize_block<kHuge>(v1, g, gd6, cd[f][2], cd[f][3]);
        const uint32_t row = m0 + f * 32 + r;
        if (kCodes && row < p.M) {
          *reinterpret_cast<uint4*>(q.codes + (size_t)row * (p.K >> 1) + kc * 32u + h * 16u) =
              make_uint4(cd[f][0], cd[f][1], cd[f][2], cd[f][3]);
          *reinterpret_cast<uint16_t*>(q.scales + (size_t)row * (p.K >> 4) + kc * 4u + h * 2u) =
              (uint16_t)(s0 | (s1 << 8));
        }
        sa[f] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(s0 | (s1 << 8), 1.0f, false);
      }
      half2v sb[FN];
#pragma unroll
      for (int f = 0; f < FN; ++f) sb[f] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(c.sb[f], 1.0f, false);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        half8 bv[FN];
#pragma unroll
        for (int f = 0; f < FN; ++f)
          bv[f] = decode8((uint32_t)c.b[f][j], j >> 1 ? __builtin_shufflevector(sb[f], sb[f], 1, 1)
                                                      : __builtin_shufflevector(sb[f], sb[f], 0, 0));
#pragma unroll
        for (int fa = 0; fa < FM; ++fa) {
          const half8 av = decode8(cd[fa][j], j >> 1 ? __builtin_shufflevector(sa[fa], sa[fa], 1, 1)
                                                     : __builtin_shufflevector(sa[fa], sa[fa], 0, 0));
#pragma unroll
          for (int fb = 0; fb < FN; ++fb)
            acc[fa][fb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bv[fb], acc[fa][fb], 0, 0, 0);
        }
      }
    };
    // Register ring of kDepth + 1 chunks: chunk i + kDepth is loaded while
    // chunk i is computed (the loop unrolled over the ring's slots).
    constexpr int kRing = kDepth + 1;
    Chunk ring[kRing];
#pragma unroll
    for (int u = 0; u < kDepth; ++u)
      if ((uint32_t)u < n_mine) load(ring[u], u);
    for (uint32_t i = 0; i < n_mine; i += kRing) {
#pragma unroll
      for (int u = 0; u < kRing; ++u) {
        if (i + u < n_mine) {
          if (i + u + kDepth < n_mine) load(ring[(u + kDepth) % kRing], i + u + kDepth);
          compute(ring[u], i + u);
        }
      }
    }
  };
  if (g > kHugeScale)
    run(std::integral_constant<bool, true>{});
  else
    run(std::integral_constant<bool, false>{});
  splitk_epilogue<KS, FM, FN, 1, kF32Out, false>(acc, part, p, alpha, y, m0, n0, wave, lane);
}

template <int KS, int FM, int FN, int kDepth>
static hipError_t launch_quant_gemm_fn(const QuantGemmArgs& q, bool dynamic, const uint8_t* w_packed,
                                       const float* w_g, void* y, GemmParams p, bool out_f32,
                                       hipStream_t stream) {
  p.tiles_m = (p.M + FM * 32 - 1) / (FM * 32);
  p.tiles_n = (p.N + FN * 32 - 1) / (FN * 32);
  const dim3 grid(p.tiles_m * p.tiles_n), block(KS * 64);
#define NVFP4_QG(D, F32, CODES)                                                                           \
  hipLaunchKernelGGL((quant_gemm_kernel<KS, FM, FN, kDepth, D, F32, CODES>), grid, block, 0, stream, q, w_packed, w_g, y, p)
  const bool codes = q.codes != nullptr;
  if (dynamic) {
    if (out_f32) { if (codes) NVFP4_QG(true, true, true); else NVFP4_QG(true, true, false); }
    else { if (codes) NVFP4_QG(true, false, true); else NVFP4_QG(true, false, false); }
  } else {
    if (out_f32) { if (codes) NVFP4_QG(false, true, true); else NVFP4_QG(false, true, false); }
    else { if (codes) NVFP4_QG(false, false, true); else NVFP4_QG(false, false, false); }
  }
#undef NVFP4_QG
  return hipGetLastError();
}

template <int KS, int FM, int FN, int kStages>
static hipError_t launch_splitk(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                                const uint8_t* w_packed, const float* w_g, void* y, GemmParams p,
                                bool out_f32, bool gate, hipStream_t stream) {
  constexpr int BM = FM * 32, BN = FN * 32;
  constexpr int kLds = KS * kStages * SplitkStage<FM, FN>::kBytes;
  static_assert(kLds >= KS * 64 * 64, "the reduction reuses the rings");
  p.tiles_m = (p.M + BM - 1) / BM;
  p.tiles_n = (p.N + BN - 1) / BN;
  const dim3 grid(p.tiles_m * p.tiles_n), block(KS * 64);
#define NVFP4_SK(F32, GATE)                                                                           \
  hipLaunchKernelGGL((gemm_splitk_kernel<KS, FM, FN, kStages, F32, GATE>), grid, block, kLds, stream, \
                     a_codes, a_scales, a_g, w_packed, w_g, y, p)
  if (gate) {
    if (out_f32) NVFP4_SK(true, true); else NVFP4_SK(false, true);
  } else {
    if (out_f32) NVFP4_SK(true, false); else NVFP4_SK(false, false);
  }
#undef NVFP4_SK
  return hipGetLastError();
}

template <int WM, int WN, int FM, int FN>
static hipError_t launch_reg(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                             const uint8_t* w_packed, const float* w_g, void* y, GemmParams p,
                             bool out_f32, bool aligned, hipStream_t stream) {
  constexpr int BM = WM * FM * 32, BN = WN * FN * 32;
  p.tiles_m = (p.M + BM - 1) / BM;
  p.tiles_n = (p.N + BN - 1) / BN;
  const dim3 grid(p.tiles_m * p.tiles_n), block(WM * WN * 64);
#define NVFP4_G(F32, AL)                                                                              \
  hipLaunchKernelGGL((gemm_reg_kernel<WM, WN, FM, FN, F32, AL>), grid, block, 0, stream, a_codes, a_scales, \
                     a_g, w_packed, w_g, y, p)
  if (out_f32) {
    if (aligned) NVFP4_G(true, true); else NVFP4_G(true, false);
  } else {
    if (aligned) NVFP4_G(false, true); else NVFP4_G(false, false);
  }
#undef NVFP4_G
  return hipGetLastError();
}

// Output columns [n_begin, n_end) (n_begin a multiple of 32).
template <class C>
static hipError_t launch_lds(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                             const uint8_t* w_packed, const float* w_g, void* y, GemmParams p,
                             uint32_t n_begin, uint32_t n_end, bool out_f32, hipStream_t stream) {
  p.n_off = n_begin;
  p.tiles_m = (p.M + C::BM - 1) / C::BM;
  p.tiles_n = (n_end - n_begin + C::BN - 1) / C::BN;
  const dim3 grid(p.tiles_m * p.tiles_n), block(C::kThreads);
  if (out_f32)
    hipLaunchKernelGGL((gemm_lds_kernel<C, true>), grid, block, C::kLdsBytes, stream, a_codes, a_scales, a_g,
                       w_packed, w_g, y, p);
  else
    hipLaunchKernelGGL((gemm_lds_kernel<C, false>), grid, block, C::kLdsBytes, stream, a_codes, a_scales, a_g,
                       w_packed, w_g, y, p);
  return hipGetLastError();
}

// Compute units of the current device (cached per device).
static uint32_t cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cached[dev] = n;
  }
  return (uint32_t)cached[dev];
}

static GemmParams gemm_params(int64_t M, int64_t K, int64_t N, const int64_t* seg_offsets, int n_seg,
                              int64_t ldy) {
  PackedDims d = packed_dims(N, K);
  GemmParams p{};
  p.M = (uint32_t)M;
  p.N = (uint32_t)N;
  p.K = (uint32_t)K;
  p.ldy = (uint32_t)ldy;
  p.chunks = (uint32_t)((K + 63) / 64);
  p.w_kc = (uint32_t)d.kc;
  p.w_scale_offset = (uint32_t)d.scale_offset;
  p.w_tiles = (uint32_t)(d.np / 32);
  p.a_code_bytes = (uint32_t)(M * K / 2);
  p.a_scale_bytes = (uint32_t)(M * K / 16);
  p.w_bytes = (uint32_t)d.bytes;
  p.n_seg = n_seg;
  for (int i = 0; i < NVFP4_SEG_TABLE; ++i)
    p.seg_off[i] = (uint32_t)seg_offsets[i <= n_seg ? i : n_seg];
  return p;
}

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                       int64_t M, int64_t K, const void* w_packed, int64_t N,
                       const int64_t* seg_offsets, int n_seg, const float* w_g, void* y,
                       int64_t ldy, bool out_f32, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  GemmParams p = gemm_params(M, K, N, seg_offsets, n_seg, ldy);
  p.y_pairs = (ldy % 2 == 0) && (reinterpret_cast<uintptr_t>(y) % 4 == 0) ? 1u : 0u;
  const uint8_t* wp = static_cast<const uint8_t*>(w_packed);
  const bool aligned = (K % 64) == 0;
  if (aligned && N <= 96)
    return launch_splitk<4, 2, 3, 3>(a_codes, a_scales, a_g, wp, w_g, y, p, out_f32, false, stream);
  if (aligned && M <= 32)
    return launch_splitk<4, 1, 2, 3>(a_codes, a_scales, a_g, wp, w_g, y, p, out_f32, false, stream);
  if (aligned) {
    // Square tiles fill whole rounds of one workgroup per CU.  When the last
    // round would be at most half full and its tiles make whole tile
    // columns, those columns run as a second launch of 256 x 128 tiles (two
    // per CU), which takes about half a round instead of a full one.
    const uint32_t tiles_m = (uint32_t)((M + LdsSquare::BM - 1) / LdsSquare::BM);
    const uint32_t tiles_n = (uint32_t)((N + LdsSquare::BN - 1) / LdsSquare::BN);
    const uint32_t n_cu = cu_count();
    const bool super = (K % 256) == 0;   // scale super-stages: 16-byte aligned, whole groups of 4 chunks
    const uint32_t rem = n_cu ? (tiles_m * tiles_n) % n_cu : 0;
    if (rem != 0 && rem <= n_cu / 2 && rem % tiles_m == 0 && rem / tiles_m < tiles_n) {
      const uint32_t n_split = (tiles_n - rem / tiles_m) * LdsSquare::BN;
      hipError_t e = super ? launch_lds<LdsSquareSuper>(a_codes, a_scales, a_g, wp, w_g, y, p, 0, n_split, out_f32, stream)
                           : launch_lds<LdsSquare>(a_codes, a_scales, a_g, wp, w_g, y, p, 0, n_split, out_f32, stream);
      if (e != hipSuccess) return e;
      return launch_lds<LdsTall>(a_codes, a_scales, a_g, wp, w_g, y, p, n_split, (uint32_t)N, out_f32, stream);
    }
    if (super)
      return launch_lds<LdsSquareSuper>(a_codes, a_scales, a_g, wp, w_g, y, p, 0, (uint32_t)N, out_f32, stream);
    return launch_lds<LdsSquare>(a_codes, a_scales, a_g, wp, w_g, y, p, 0, (uint32_t)N, out_f32, stream);
  }
  return launch_reg<2, 2, 4, 4>(a_codes, a_scales, a_g, wp, w_g, y, p, out_f32, aligned, stream);
}

hipError_t launch_gemm_gdn_gates(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                                 int64_t M, int64_t K, const void* w_packed, int64_t H, const float* w_g,
                                 const float* a_log, const float* dt_bias, void* y, int64_t ldy,
                                 bool out_f32, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int64_t offs[3] = {0, H, 2 * H};
  GemmParams p = gemm_params(M, K, 2 * H, offs, 2, ldy);
  p.gate_a_log = a_log;
  p.gate_dt_bias = dt_bias;
  p.gate_h = (uint32_t)H;
  return launch_splitk<4, 2, 3, 3>(a_codes, a_scales, a_g, static_cast<const uint8_t*>(w_packed), w_g, y, p,
                                   out_f32, true, stream);
}

hipError_t launch_quant_gemm(const void* x, int64_t M, int64_t K, int64_t ldx, float* g_enc, bool dynamic,
                             float* partial, const void* w_packed, int64_t N, const int64_t* seg_offsets,
                             int n_seg, const float* w_g, uint8_t* codes, uint8_t* scales, void* y, int64_t ldy,
                             bool out_f32, hipStream_t stream) {
  if (M == 0) {   // G as the quantizer writes it for an empty tensor
    if (!dynamic) return hipSuccess;
    return launch_act_quant(x, 0, K, ldx, codes, scales, g_enc, true, partial, stream);
  }
  QuantGemmArgs q{};
  q.x = static_cast<const uint16_t*>(x);
  q.x_bytes = (uint32_t)(M * ldx * 2);
  q.ldx_bytes = (uint32_t)(ldx * 2);
  q.g_enc = g_enc;
  q.partial = partial;
  q.codes = codes;
  q.scales = scales;
  if (dynamic) {
    int n_partial = 0;
    hipError_t e = launch_act_amax(x, M, K, ldx, partial, &n_partial, stream);
    if (e != hipSuccess) return e;
    q.n_partial = (uint32_t)n_partial;
  }
  GemmParams p = gemm_params(M, K, N, seg_offsets, n_seg, ldy);
  const uint8_t* wp = static_cast<const uint8_t*>(w_packed);
  if (N <= 96) return launch_quant_gemm_fn<4, 2, 3, 1>(q, dynamic, wp, w_g, y, p, out_f32, stream);
  return launch_quant_gemm_fn<4, 1, 4, 1>(q, dynamic, wp, w_g, y, p, out_f32, stream);
}

}  // namespace nvfp4
