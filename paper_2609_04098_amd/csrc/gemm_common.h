// Shared device code and host-side plumbing of the NVFP4 GEMM kernels
// (gemm_lds_*.hip, gemm_splitk.hip, gemm_reg.hip, quant_gemm.hip; the host
// dispatch is in gemm.hip).
//
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
//    reduction, each streaming its weight chunks through a private LDS ring
//    and the activation, whole 128-byte row lines of 4 chunks, through a
//    ring shared by the workgroup; the partial sums meet in LDS.
//  * gemm_reg_kernel (K % 64 != 0, N > 96): operands go straight from global
//    memory to registers one chunk ahead; per-block masking of the scales
//    handles a K tail.
// All remap workgroups so that each XCD (its own L2) runs a contiguous,
// M-grouped range of tiles; out-of-range rows/columns read zeros through the
// buffer bounds and are not stored.
#include <hip/hip_runtime.h>
#pragma once

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
  // BF16 output at least as large as the MALL: the LDS kernel's staged
  // stores are non-temporal (the output cannot stay cached, and its lines
  // go to HBM while the GEMM leaves HBM idle instead of being written back
  // when the next kernel's reads evict them).
  uint32_t y_stream;
  // K split across workgroups (LDS kernel, FP32 output only): k_parts = 2
  // runs every tile twice, workgroup 2t + j on chunks [j * chunks, (j + 1) *
  // chunks) writing its partial sums at y + j * part_stride floats.
  uint32_t k_parts, part_stride;
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
// Cache-policy operand of a buffer load: device scope (coherent across the
// XCDs' L2 caches).
constexpr int kDeviceScope = 16;
template <int kAux = 0>
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, uint8_t* dst, uint32_t voffset, uint32_t soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (NVFP4_LDS void*)dst, 16, voffset, soffset, 0, kAux);
}
template <int kAux = 0>
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t rs, uint8_t* dst, uint32_t voffset, uint32_t soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (NVFP4_LDS void*)dst, 4, voffset, soffset, 0, kAux);
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
__device__ __forceinline__ void tile_of(const GemmParams& p, uint32_t& tm, uint32_t& tn,
                                        uint32_t pid0 = blockIdx.x) {
  const uint32_t total = p.tiles_m * p.tiles_n;
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
constexpr int kLgkm0Mask = ~(15 << 8);        // AND into a vmcnt_imm wait: also lgkmcnt(0)
}  // namespace lds

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

// Shared activation stage of the split-K kernel (streamed activation, FM
// fragments of 32 rows): one 128-byte line group per row (4 chunks of codes)
// as FM * 4 slices of 8 rows (1 KB images), then per slice the 16 bytes of
// scales of its 8 rows in a 260-byte slot (128 bytes of scales, 128 bytes of
// zeros from the lanes without a row, 4 bytes that shift the next slot's
// banks).  Each of the 4 waves loads FM slices.
template <int FM>
struct SplitkAGroup {
  static constexpr int kSlices = 4 * FM, kSlicesPerWave = FM;
  static constexpr int kScaleBase = kSlices * 1024, kScaleSlot = 260;
  static constexpr int kBytes = (kScaleBase + kSlices * kScaleSlot + 15) / 16 * 16;
  static constexpr int kLoadsPerWave = 2 * kSlicesPerWave;
};

// LDS of the split-K kernel: KS private weight rings, then the shared
// activation ring (streamed activation) or nothing (the fused quantizer puts
// its activation after the rings).
template <int KS, int FM, int FN, int kStages, bool kAShared>
constexpr int splitk_ring_bytes() {
  return KS * kStages * SplitkStage<0, FN>::kBytes + (kAShared ? kStages * SplitkAGroup<FM>::kBytes : 0);
}

// Operands of one GEMM call (device pointers), as passed to the launchers.
struct GemmOperands {
  const uint8_t* a_codes;
  const uint8_t* a_scales;
  const float* a_g;
  const uint8_t* w_packed;
  const float* w_g;
  void* y;
};

inline GemmParams gemm_params(int64_t M, int64_t K, int64_t N, const int64_t* seg_offsets, int n_seg,
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
  p.k_parts = 1;
  p.part_stride = 0;
  p.n_seg = n_seg;
  for (int i = 0; i < NVFP4_SEG_TABLE; ++i)
    p.seg_off[i] = (uint32_t)seg_offsets[i <= n_seg ? i : n_seg];
  return p;
}

// MALL (last-level memory-side cache) of the MI355X.
constexpr uint64_t kMallBytes = 256ull << 20;

// Side of the square prefill tile (gemm_lds_kernel<LdsSquare*>).
constexpr uint32_t kSquareTile = 256;

// The kernels one nvfp4_gemm call launches: `first` over output columns
// [0, n_split), then `second` (if any) over [n_split, N).
struct GemmPlan {
  enum Kind { kNone = 0, kLdsSquare, kLdsSuper, kLdsTall, kSplitkNarrow, kSplitkDecode, kReg, kLdsSuperHalves,
              kSplitkDecodeFew };
  int first, second;
  uint32_t n_split;
};
// with_ws: the caller provides gemm_workspace_bytes of workspace (the last
// round's tile columns may then run as two K halves on twice the CUs).
GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, uint32_t n_cu, bool with_ws);
size_t plan_workspace_bytes(const GemmPlan& g, int64_t M, int64_t N);
const char* gemm_kernel_name(int kind);

// Launchers of the kernel families (each in its own translation unit).
// Prefill tiles over output columns [n_begin, n_end) (n_begin a multiple of 32).
hipError_t launch_lds_square(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end, bool out_f32,
                             hipStream_t stream);
hipError_t launch_lds_super_bf16(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end,
                                 hipStream_t stream);
hipError_t launch_lds_super_f32(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end,
                                hipStream_t stream);
// The same kernel over columns [n_begin, n_end) with the K range split in
// two halves (p.chunks % 8 == 0): FP32 partial sums (segment-scaled) to
// parts[2][M][halves_row(n_end - n_begin)]; sum_halves then forms Y.
inline uint32_t halves_row(uint32_t width) { return (width + 3u) & ~3u; }
hipError_t launch_lds_super_halves(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end,
                                   float* parts, hipStream_t stream);
hipError_t launch_sum_halves(const float* parts, uint32_t M, uint32_t width, void* y, uint32_t ldy, uint32_t col0,
                             bool out_f32, hipStream_t stream);
hipError_t launch_lds_tall(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end, bool out_f32,
                           hipStream_t stream);
// Split-K: 64 x 96 tiles (N <= 96, optional GDN gate epilogue); M <= 32:
// 32 x 32 tiles (M <= 8) or 32 x 64 tiles.
hipError_t launch_splitk_narrow(const GemmOperands& o, GemmParams p, bool out_f32, bool gate, hipStream_t stream);
hipError_t launch_splitk_decode(const GemmOperands& o, GemmParams p, bool out_f32, hipStream_t stream);
// Largest activation (in 16-element blocks) the fused decode launch
// quantizes inside every workgroup: 1024 blocks = M * K <= 16384 elements.
constexpr uint32_t kDecodeFuseMaxBlocks = 1024;
// Activation quantization fused in front of the M <= 32 split-K GEMM, one
// launch, with the whole quantized activation held in LDS (see
// gemm_splitk.hip); decode_quant_lds_bytes(M, K) is the dynamic LDS it takes
// (the rings; the activation sits in a static 9 KB array).
struct DecodeQuantArgs {
  const uint16_t* x;        // bf16 [M x K], row stride ldx elements
  uint32_t ldx;
  float* g_enc;             // written (dynamic, by workgroup 0) or read (given G)
  uint8_t* codes;           // optional outputs ([M x K/2], [M x K/16]), written by workgroup 0
  uint8_t* scales;
};
size_t decode_quant_lds_bytes(int64_t M, int64_t K);
hipError_t launch_decode_quant_gemm(const GemmOperands& o, GemmParams p, const DecodeQuantArgs& q, bool dynamic,
                                    bool out_f32, hipStream_t stream);
// Register path (K % 64 != 0).
hipError_t launch_reg_square(const GemmOperands& o, GemmParams p, bool out_f32, bool aligned, hipStream_t stream);

}  // namespace nvfp4
