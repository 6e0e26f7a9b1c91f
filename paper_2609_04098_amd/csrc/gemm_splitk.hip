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
                     o.a_codes, o.a_scales, o.a_g, o.w_packed, o.w_g, o.y, p)
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

}  // namespace nvfp4
