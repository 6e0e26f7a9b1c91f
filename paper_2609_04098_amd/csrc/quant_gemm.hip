// Activation quantization fused into the NVFP4 GEMM (nvfp4_quantize_gemm):
// the narrow-output kernel below (N <= 128), and the host side of the fused
// decode path (M <= 32, the split-K kernel's fused prologue).
#include "gemm_common.h"

namespace nvfp4 {

// ------------------------------------------- fused quantize + tall-skinny GEMM
//
// For narrow outputs (N <= 128: the gate projections), the activation is
// quantized inside the GEMM: each lane takes the 32 bf16 values it supplies
// to the MFMA (row r, reduction indices [32h, 32h + 32) of the chunk: two
// whole blocks), quantizes them with the same device code as the stand-alone
// quantizer (so the codes are identical), optionally stores the codes and
// scales, and feeds the decoded values to the MFMA; X is read once and the
// codes never travel through memory.  Tile: FM x 32 rows x FN fragments, the
// KS waves of a workgroup split the reduction (wave w takes chunks w,
// w + KS, ...), and the partial sums meet in LDS (splitk_epilogue).  G_A is read (static) or formed from
// the amax pass's partial maxima (dynamic; workgroup 0 writes it out), and
// the epilogue uses the value, not the memory.  K % 64 == 0.
//
// X moves global -> LDS by direct-to-LDS loads that read whole 128-byte row
// lines (one wave-wide load: 8 rows of the chunk), into two per-wave slots
// (the chunks i + 1 and i + 2 in flight while chunk i is quantized), and
// each lane then reads its 64 bytes back from LDS.  Loading a lane's own 64
// bytes straight into registers touches 32 lines per load, holds two
// chunks of X in registers, and measured 2-3% slower at 32768 x 96 x 5120.
// The weight goes straight to registers, three chunks deep.
struct QuantGemmArgs {
  const uint16_t* x;
  uint32_t x_bytes, ldx_bytes;
  float* g_enc;
  const float* partial;
  uint32_t n_partial;
  uint8_t* codes;
  uint8_t* scales;
};

// One X slot: the chunk's FM * 4 images of 8 rows x 128 bytes.
template <int FM>
constexpr int quant_gemm_xslot_bytes() { return FM * 4 * 1024; }

template <int KS, int FM, int FN, bool kDynamic, bool kF32Out, bool kCodes>
__global__ __launch_bounds__(KS * 64, 2) void quant_gemm_kernel(QuantGemmArgs q, const uint8_t* __restrict__ w_packed,
                                                            const float* __restrict__ w_g, void* __restrict__ y,
                                                            GemmParams p) {
  constexpr int kXSlot = quant_gemm_xslot_bytes<FM>();
  static_assert(2 * kXSlot >= 64 * 64, "the partial sums reuse the slots");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
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
  // X image t = 4 f + j holds rows 32 f + 8 j .. + 7: lane l loads 16-byte
  // piece (l % 8) ^ (l / 8) ^ (t % 8) of row 32 f + 8 j + l / 8 into slot l,
  // and lane (h, r) finds piece 4 h + u of its row r (image 4 f + r / 8) at
  // slot (r % 8) * 8 + ((4 h + u) ^ (r % 8) ^ (t % 8)): the 16 lanes of one
  // LDS read hit distinct banks.
  const __amdgpu_buffer_rsrc_t rx = rsrc(q.x, q.x_bytes);
  uint32_t x_off[FM][4], x_rd[FM][4], c_off[FM], s_off[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t t = 4 * f + j, row = m0 + 32 * f + 8 * j + (lane >> 3);
      const uint32_t piece = (lane & 7) ^ (lane >> 3) ^ (t & 7);
      x_off[f][j] = row < p.M ? row * q.ldx_bytes + piece * 16u : kOOB;
      const uint32_t tr = 4 * f + (r >> 3), rr = r & 7;
      x_rd[f][j] = tr * 1024u + (rr * 8u + ((4 * h + j) ^ rr ^ (tr & 7))) * 16u;
    }
    const uint32_t row = m0 + f * 32 + r;
    c_off[f] = row < p.M ? row * (p.K >> 1) + h * 16u : kOOB;
    s_off[f] = row < p.M ? row * (p.K >> 4) + h * 2u : kOOB;
  }
  uint8_t* xs = smem + wave * (2 * kXSlot);
  const __amdgpu_buffer_rsrc_t rc = rsrc(q.codes, p.a_code_bytes);
  const __amdgpu_buffer_rsrc_t rsc = rsrc(q.scales, p.a_scale_bytes);
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
  struct WRegs {
    int4v b[FN];
    uint32_t sb[FN];
  };
  // Chunk i of this wave: X into slot i % 2, the weight into registers.
  auto load = [&](WRegs& w, uint32_t i) {
    const uint32_t kc = wave + KS * i;
    uint8_t* dst = xs + (i & 1) * kXSlot;
#pragma unroll
    for (int f = 0; f < FM; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j) dma16(rx, dst + (4 * f + j) * 1024, x_off[f][j], kc * 128u);
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      w.b[f] = __builtin_amdgcn_raw_buffer_load_b128(rb, b_off[f], kc * 1024u, 0);
      w.sb[f] = __builtin_amdgcn_raw_buffer_load_b16(rbs, bs_off[f], kc * 128u, 0);
    }
  };
  constexpr int kLoads = FM * 4 + 2 * FN;                    // loads per chunk, in issue order
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
        const uint32_t s0 = quantize_block<kHuge, false>(v0, g, gd6, cd[f][0], cd[f][1]);
        const uint32_t s1 = quantize_block<kHuge, false>(v1, g, gd6, cd[f][2], cd[f][3]);
        if (kCodes) {
          // Buffer stores: the lane's offset is fixed, the chunk goes in the
          // scalar offset; rows >= M have offsets past the buffers (dropped).
          __builtin_amdgcn_raw_buffer_store_b128(int4v{(int)cd[f][0], (int)cd[f][1], (int)cd[f][2], (int)cd[f][3]},
                                                 rc, c_off[f], kc * 32u, 0);
          __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(s0 | (s1 << 8)), rsc, s_off[f], kc * 4u, 0);
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
    // Chunks i + 1 and i + 2 are in flight while chunk i is computed; the
    // weight registers rotate over three sets (the loop unrolled over them),
    // the X slot of chunk i is refilled once its LDS reads have returned.
    WRegs wr[3];
    if (n_mine > 0) load(wr[0], 0);
    if (n_mine > 1) load(wr[1], 1);
    for (uint32_t i = 0; i < n_mine; i += 3) {
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const uint32_t ii = i + u;
        if (ii < n_mine) {
          if (ii + 1 < n_mine)
            __builtin_amdgcn_s_waitcnt(lds::vmcnt_imm(kLoads));   // chunk ii landed
          else
            __builtin_amdgcn_s_waitcnt(lds::vmcnt_imm(0));
          Chunk c;
          const uint8_t* src = xs + (ii & 1) * kXSlot;
#pragma unroll
          for (int f = 0; f < FM; ++f)
#pragma unroll
            for (int j = 0; j < 4; ++j) c.x[f][j] = *(const int4v*)(src + x_rd[f][j]);
#pragma unroll
          for (int f = 0; f < FN; ++f) {
            c.b[f] = wr[u].b[f];
            c.sb[f] = wr[u].sb[f];
          }
          __builtin_amdgcn_s_waitcnt(lds::kWaitLgkm0);            // slot ii % 2 read
          if (ii + 2 < n_mine) load(wr[(u + 2) % 3], ii + 2);
          compute(c, ii);
        }
      }
    }
  };
  if (g > kHugeScale)
    run(std::integral_constant<bool, true>{});
  else
    run(std::integral_constant<bool, false>{});
  // The partial sums reuse the X slots (every load has landed: the last
  // chunk waited for all of them).
  __syncthreads();
  splitk_epilogue<KS, FM, FN, 1, kF32Out, false>(acc, reinterpret_cast<floatx16*>(smem), p, alpha, y, m0, n0, wave,
                                                 lane);
}

template <int KS, int FM, int FN>
static hipError_t launch_quant_gemm_fn(const QuantGemmArgs& q, bool dynamic, const uint8_t* w_packed,
                                       const float* w_g, void* y, GemmParams p, bool out_f32,
                                       hipStream_t stream) {
  p.tiles_m = (p.M + FM * 32 - 1) / (FM * 32);
  p.tiles_n = (p.N + FN * 32 - 1) / (FN * 32);
  const dim3 grid(p.tiles_m * p.tiles_n), block(KS * 64);
  constexpr uint32_t kLds = KS * 2 * quant_gemm_xslot_bytes<FM>();
  static_assert(2 * kLds <= 160 * 1024 - 64, "two workgroups per CU");
#define NVFP4_QG(D, F32, CODES)                                                                           \
  hipLaunchKernelGGL((quant_gemm_kernel<KS, FM, FN, D, F32, CODES>), grid, block, kLds, stream, q, w_packed, w_g, y, p)
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

namespace {

size_t align16(size_t v) { return (v + 15) & ~(size_t)15; }

// The fused decode kernel quantizes all of X in every workgroup (there is
// no hand-off between workgroups), so it pays off only while X is a few
// tokens: up to M * K = 16384 elements (3 tokens of width 5120) it beats
// the quantizer launch in front of the GEMM (1 token: 30.2 vs 32.4 us on
// the gate/up weight read from HBM); at 7 tokens the repeated quantization
// already costs more than the launch (43.6 vs 36.7 us).
constexpr int64_t kDecodeFuseMaxElems = 16 * (int64_t)kDecodeFuseMaxBlocks;

}  // namespace

bool quant_gemm_uses_decode_path(int64_t M, int64_t N) { return M >= 1 && M <= 32 && N > 128; }

// Workspace of nvfp4_quantize_gemm: the partial maxima of the amax pass
// (kActScratchBytes); on the decode path also room for the quantized
// activation (codes, then scales) when it runs as two launches.
size_t quant_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  size_t bytes = kActScratchBytes;
  if (quant_gemm_uses_decode_path(M, N)) bytes += align16((size_t)(M * K / 2)) + align16((size_t)(M * K / 16));
  return bytes;
}

hipError_t launch_quant_gemm(const void* x, int64_t M, int64_t K, int64_t ldx, float* g_enc, bool dynamic,
                             void* workspace, const void* w_packed, int64_t N, const int64_t* seg_offsets,
                             int n_seg, const float* w_g, uint8_t* codes, uint8_t* scales, void* y, int64_t ldy,
                             bool out_f32, hipStream_t stream) {
  float* partial = static_cast<float*>(workspace);
  if (M == 0) {   // G as the quantizer writes it for an empty tensor
    if (!dynamic) return hipSuccess;
    return launch_act_quant(x, 0, K, ldx, codes, scales, g_enc, true, partial, stream);
  }
  GemmParams p = gemm_params(M, K, N, seg_offsets, n_seg, ldy);
  const uint8_t* wp = static_cast<const uint8_t*>(w_packed);
  if (quant_gemm_uses_decode_path(M, N)) {
    if (M * K <= kDecodeFuseMaxElems) {
      // One launch: every workgroup quantizes X into its LDS.
      const DecodeQuantArgs dq{static_cast<const uint16_t*>(x), (uint32_t)ldx, g_enc, codes, scales};
      const GemmOperands o{codes, scales, g_enc, wp, w_g, y};
      return launch_decode_quant_gemm(o, p, dq, dynamic, out_f32, stream);
    }
    // Larger activations: the quantizer, then the same GEMM kernel reading
    // the codes from memory (the caller's buffers or the workspace).
    uint8_t* ws = static_cast<uint8_t*>(workspace) + kActScratchBytes;
    uint8_t* a_codes = codes != nullptr ? codes : ws;
    uint8_t* a_scales = scales != nullptr ? scales : ws + align16((size_t)(M * K / 2));
    hipError_t e = launch_act_quant(x, M, K, ldx, a_codes, a_scales, g_enc, dynamic, partial, stream);
    if (e != hipSuccess) return e;
    const GemmOperands o{a_codes, a_scales, g_enc, wp, w_g, y};
    return launch_splitk_decode(o, p, out_f32, stream);
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
  if (N <= 96) return launch_quant_gemm_fn<4, 2, 3>(q, dynamic, wp, w_g, y, p, out_f32, stream);
  return launch_quant_gemm_fn<4, 1, 4>(q, dynamic, wp, w_g, y, p, out_f32, stream);
}

}  // namespace nvfp4
