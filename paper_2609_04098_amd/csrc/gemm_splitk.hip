// Split-K NVFP4 GEMM for outputs with few 32 x 32 tiles (tall-skinny gate
// projections, decode-shaped calls).
#include "gemm_common.h"

namespace nvfp4 {

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

// Activation quantization fused in front of the split-K GEMM, one launch,
// for decode shapes whose whole activation fits in LDS (kQuant = 1 with a
// given G, 2 with the dynamic G).  Every workgroup reads all of X (a few KB
// to a few tens of KB, from L2 after the first workgroup), takes the global
// maximum itself in dynamic mode (the maximum is order-free, so every
// workgroup forms the same G), quantizes every block with the stand-alone
// quantizer's device code into LDS, and the GEMM then reads its activation
// fragments from LDS instead of streaming them: one launch, no hand-off
// between workgroups, and the results of nvfp4_quantize_act + nvfp4_gemm
// bit for bit (same codes, same summation order).  Workgroup 0 also writes
// G and, when asked for, the codes and scales.

// Maximum over the workgroup (kThreads threads) of a non-negative value.
template <int kThreads>
__device__ __forceinline__ uint32_t wg_max_u32(uint32_t v, uint32_t* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = __shfl_xor(v, off, 64);
    v = v > o ? v : o;
  }
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t r = red[0];
#pragma unroll
  for (int w = 1; w < kThreads / 64; ++w) r = r > red[w] ? r : red[w];
  __syncthreads();
  return r;
}

// The 8 dwords (16 bf16) of block b of X (row-major blocks, bpr per row).
__device__ __forceinline__ void load_x_block(const DecodeQuantArgs& q, uint32_t b, uint32_t bpr, uint32_t v[8]) {
  const uint32_t row = b / bpr, col = b - row * bpr;
  const uint4* src = reinterpret_cast<const uint4*>(q.x + (size_t)row * q.ldx) + 2 * col;
  const uint4 d0 = src[0], d1 = src[1];
  v[0] = d0.x; v[1] = d0.y; v[2] = d0.z; v[3] = d0.w;
  v[4] = d1.x; v[5] = d1.y; v[6] = d1.z; v[7] = d1.w;
}

// Quantize all of X into the LDS activation (codes [M][K/2], then scales
// [M][K/16]); returns G.
template <int kThreads, bool kDynamic>
__device__ float quantize_into_lds(const DecodeQuantArgs& q, const GemmParams& p, uint8_t* lds_codes,
                                   uint8_t* lds_scales, uint32_t* red) {
  const uint32_t bpr = p.K >> 4, n_blocks = p.M * bpr;
  float g;
  if (kDynamic) {
    uint32_t m = 0;
    for (uint32_t b = threadIdx.x; b < n_blocks; b += kThreads) {
      uint32_t v[8];
      load_x_block(q, b, bpr, v);
      const uint32_t a = __float_as_uint(block_amax(v));
      m = m > a ? m : a;                     // non-negative floats order as integers
    }
    g = global_scale(__uint_as_float(wg_max_u32<kThreads>(m, red)));
    if (blockIdx.x == 0 && threadIdx.x == 0) *q.g_enc = g;
  } else {
    g = *q.g_enc;
  }
  const float gd6 = g * (1.0f / 6.0f);
  const bool out = q.codes != nullptr && blockIdx.x == 0;
  for (uint32_t b = threadIdx.x; b < n_blocks; b += kThreads) {
    uint32_t v[8], c0, c1, sc;
    load_x_block(q, b, bpr, v);
    if (g > kHugeScale)
      sc = quantize_block<true>(v, g, gd6, c0, c1);
    else
      sc = quantize_block<false>(v, g, gd6, c0, c1);
    reinterpret_cast<uint2*>(lds_codes)[b] = make_uint2(c0, c1);
    lds_scales[b] = (uint8_t)sc;
    if (out) {
      reinterpret_cast<uint2*>(q.codes)[b] = make_uint2(c0, c1);
      q.scales[b] = (uint8_t)sc;
    }
  }
  __syncthreads();
  return g;
}

template <int KS, int FM, int FN, int kStages, bool kF32Out, bool kGate, int kQuant = 0>
__global__ __launch_bounds__(KS * 64, 2) void gemm_splitk_kernel(const uint8_t* __restrict__ a_codes,
                                                             const uint8_t* __restrict__ a_scales,
                                                             const float* __restrict__ a_g,
                                                             const uint8_t* __restrict__ w_packed,
                                                             const float* __restrict__ w_g,
                                                             void* __restrict__ y, GemmParams p,
                                                             DecodeQuantArgs q) {
  constexpr int BM = FM * 32, BN = FN * 32;
  // With the fused quantizer the activation sits in LDS and the ring
  // carries only the weight.
  constexpr bool kALds = kQuant != 0;
  static_assert(!kALds || FM == 1, "LDS-resident activation: one 32-row fragment");
  using L = SplitkStage<kALds ? 0 : FM, FN>;
  constexpr int kFrags = FM + FN;
  constexpr int kWOff = kALds ? 0 : FM;                      // first weight slot of a stage
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
  uint32_t a_off[FM], as_off[L::kPairsA > 0 ? L::kPairsA : 1], b_off[FN], bs_off[L::kPairsB];
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
  const __amdgpu_buffer_rsrc_t ra = rsrc(a_codes, p.a_code_bytes);
  const __amdgpu_buffer_rsrc_t rs = rsrc(a_scales, p.a_scale_bytes);
  const __amdgpu_buffer_rsrc_t rb = rsrc(w_packed, p.w_scale_offset);
  const __amdgpu_buffer_rsrc_t rbs = rsrc(w_scales, w_scale_bytes);
  // DMA of this wave's i-th chunk into stage i % kStages.  (Prologue loads
  // of chunks past the end of K, when K is short, re-load the last chunk so
  // that every address stays inside its tensor; they are never read.)
  auto issue_a = [&](uint32_t i) {
    if constexpr (!kALds) {
      const uint32_t kc = wave + KS * i;
      const uint32_t kq = kc < p.chunks ? kc : p.chunks - 1;
      uint8_t* st = ring + (i % kStages) * kStageBytes;
#pragma unroll
      for (int f = 0; f < FM; ++f) dma16(ra, st + f * 1024, a_off[f], kq * 32u);
#pragma unroll
      for (int j = 0; j < L::kPairsA; ++j) dma4(rs, st + kScaleA + j * 256, as_off[j], kq * 4u);
    }
  };
  auto issue_w = [&](uint32_t i) {
    const uint32_t kc = wave + KS * i;
    const uint32_t kq = kc < p.chunks ? kc : p.chunks - 1;
    uint8_t* st = ring + (i % kStages) * kStageBytes;
#pragma unroll
    for (int f = 0; f < FN; ++f) dma16(rb, st + (kWOff + f) * 1024, b_off[f], kq * 1024u);
#pragma unroll
    for (int j = 0; j < L::kPairsB; ++j) dma4(rbs, st + kScaleB + j * 256, bs_off[j], kq * 128u);
  };
  auto issue = [&](uint32_t i) {
    issue_a(i);
    issue_w(i);
  };

  struct Regs {
    int4v c[kFrags];
    uint32_t s[kFrags];
  };
  // LDS-resident activation (fused quantizer): codes [M][K/2], then scales
  // [M][K/16], after the rings; rows >= M are zero operands.
  const uint8_t* a_lds = smem + KS * kStages * kStageBytes;
  const uint8_t* as_lds = a_lds + p.M * (p.K >> 1);
  auto read_stage = [&](Regs& R, uint32_t i) {
    const uint8_t* st = ring + (i % kStages) * kStageBytes;
#pragma unroll
    for (int f = 0; f < kFrags; ++f) {
      if (kALds && f < FM) {
        const uint32_t kc = wave + KS * i;
        const bool live = r < p.M && kc < p.chunks;
        R.c[f] = live ? *(const int4v*)(a_lds + r * (p.K >> 1) + kc * 32 + h * 16) : int4v{0, 0, 0, 0};
        R.s[f] = live ? *(const uint32_t*)(as_lds + r * (p.K >> 4) + kc * 4) : 0u;
      } else {
        R.c[f] = *(const int4v*)(st + (f - FM + kWOff) * 1024 + lane * 16);
        R.s[f] = *(const uint32_t*)(st + (f < FM ? kScaleA + f * 128 : kScaleB + (f - FM) * 128) + r * 4);
      }
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

  float alpha[FN];
  if constexpr (kQuant != 0) {
    // The weight's first stages do not depend on the activation: their
    // loads fly while the workgroup quantizes X into LDS.
    __shared__ uint32_t red[KS];
#pragma unroll
    for (int s = 0; s < kStages; ++s) issue_w(s);
    uint8_t* a_dst = smem + KS * kStages * kStageBytes;
    const float ga = quantize_into_lds<KS * 64, kQuant == 2>(q, p, a_dst, a_dst + p.M * (p.K >> 1), red);
    segment_alpha<FN>(p, ga, w_g, n0, r, alpha);
    __builtin_amdgcn_s_waitcnt(kWaitFirst);
  } else {
    segment_alpha<FN>(p, *a_g, w_g, n0, r, alpha);
#pragma unroll
    for (int s = 0; s < kStages; ++s) issue(s);
    __builtin_amdgcn_s_waitcnt(kWaitFirst);
  }
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

template <int KS, int FM, int FN, int kStages>
static hipError_t launch_splitk(const GemmOperands& o, GemmParams p, bool out_f32, bool gate, hipStream_t stream) {
  constexpr int BM = FM * 32, BN = FN * 32;
  constexpr int kLds = KS * kStages * SplitkStage<FM, FN>::kBytes;
  static_assert(kLds >= KS * 64 * 64, "the reduction reuses the rings");
  p.tiles_m = (p.M + BM - 1) / BM;
  p.tiles_n = (p.N + BN - 1) / BN;
  const dim3 grid(p.tiles_m * p.tiles_n), block(KS * 64);
#define NVFP4_SK(F32, GATE)                                                                           \
  hipLaunchKernelGGL((gemm_splitk_kernel<KS, FM, FN, kStages, F32, GATE>), grid, block, kLds, stream, \
                     o.a_codes, o.a_scales, o.a_g, o.w_packed, o.w_g, o.y, p, DecodeQuantArgs{})
  if (gate) {
    if (out_f32) NVFP4_SK(true, true); else NVFP4_SK(false, true);
  } else {
    if (out_f32) NVFP4_SK(true, false); else NVFP4_SK(false, false);
  }
#undef NVFP4_SK
  return hipGetLastError();
}

hipError_t launch_splitk_narrow(const GemmOperands& o, GemmParams p, bool out_f32, bool gate, hipStream_t stream) {
  return launch_splitk<4, 2, 3, 3>(o, p, out_f32, gate, stream);
}

hipError_t launch_splitk_decode(const GemmOperands& o, GemmParams p, bool out_f32, hipStream_t stream) {
  return launch_splitk<4, 1, 2, 3>(o, p, out_f32, false, stream);
}

size_t decode_quant_lds_bytes(int64_t M, int64_t K) {
  return (size_t)(4 * 3 * SplitkStage<0, 2>::kBytes) + (size_t)(M * K / 2 + M * K / 16);
}

hipError_t launch_decode_quant_gemm(const GemmOperands& o, GemmParams p, const DecodeQuantArgs& q, bool dynamic,
                                    bool out_f32, hipStream_t stream) {
  constexpr int KS = 4, FM = 1, FN = 2, kStages = 3;
  constexpr int kRing = KS * kStages * SplitkStage<0, FN>::kBytes;
  static_assert(kRing >= KS * 64 * 64, "the reduction reuses the rings");
  const size_t lds = decode_quant_lds_bytes(p.M, p.K);
  p.tiles_m = 1;
  p.tiles_n = (p.N + FN * 32 - 1) / (FN * 32);
  const dim3 grid(p.tiles_n), block(KS * 64);
#define NVFP4_DQ(F32, Q)                                                                                   \
  hipLaunchKernelGGL((gemm_splitk_kernel<KS, FM, FN, kStages, F32, false, Q>), grid, block, (uint32_t)lds, stream, \
                     o.a_codes, o.a_scales, o.a_g, o.w_packed, o.w_g, o.y, p, q)
  if (dynamic) {
    if (out_f32) NVFP4_DQ(true, 2); else NVFP4_DQ(false, 2);
  } else {
    if (out_f32) NVFP4_DQ(true, 1); else NVFP4_DQ(false, 1);
  }
#undef NVFP4_DQ
  return hipGetLastError();
}

}  // namespace nvfp4
