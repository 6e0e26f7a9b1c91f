// Split-K NVFP4 GEMM for outputs with few 32 x 32 tiles (tall-skinny gate
// projections, decode-shaped calls).
#include "gemm_common.h"

namespace nvfp4 {

// ----------------------------------------------------------- split-K path
//
// Shapes whose output has too few 32 x 32 tiles to give every SIMD two waves
// (N <= 96: the tall-skinny gate projections; M <= 32: decode-shaped calls,
// weight-bandwidth-bound): the KS = 4 waves of a workgroup share one FM x FN
// fragment tile and split its reduction, wave w taking chunks w, w + 4, ...,
// so that at step i the workgroup consumes chunks 4i .. 4i + 3.
// The weight fragments of a wave's chunk go through a private LDS ring
// (direct-to-LDS loads, refilled as soon as the wave has read a stage).
// The activation of a step, the same rows for all four waves, is one
// 128-byte line group per row (4 chunks x 32 bytes of codes, 16 bytes of
// scales), which the waves load together, a quarter each, into a ring shared
// by the workgroup: a wave-wide load then covers 8 whole rows instead of 32
// rows x 16 bytes, and a row's line is fetched once per workgroup instead of
// once per wave (the per-chunk loads of 32-byte row pieces took 3-4 times
// as many memory requests as the weight).  One barrier per step: after it
// every wave's share of the next step has landed and every wave has read
// the stage about to be refilled.  Each wave reads the next chunk's raw
// fragments from LDS while it decodes and multiplies the current one, and
// the partial sums meet in LDS at the end; fragment f is summed in wave
// order (deterministic) and stored by wave f % KS.  Requires K % 64 == 0.

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

// Workgroup barrier for LDS data only: waits for this wave's LDS accesses,
// not for its outstanding global loads (__syncthreads' fence would also wait
// for the weight ring's DMA issued before the activation is quantized).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(lds::kWaitLgkm0);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Maximum over the workgroup (kThreads threads) of a non-negative value.
template <int kThreads>
__device__ __forceinline__ uint32_t wg_max_u32(uint32_t v, uint32_t* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = __shfl_xor(v, off, 64);
    v = v > o ? v : o;
  }
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  lds_barrier();
  uint32_t r = red[0];
#pragma unroll
  for (int w = 1; w < kThreads / 64; ++w) r = r > red[w] ? r : red[w];
  lds_barrier();
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
// [M][K/16]); returns G.  X has at most kDecodeFuseMaxBlocks blocks (the
// launcher's bound): each thread loads its blocks once (load_x_slots, issued
// before the weight's first ring stages, so that waiting for X does not
// wait for them too: the memory counter counts loads in issue order) and
// keeps them in registers from the maximum to the quantization.
template <int kThreads>
struct XSlots {
  static constexpr int kSlots = kDecodeFuseMaxBlocks / kThreads;
  static_assert(kSlots * kThreads == kDecodeFuseMaxBlocks, "blocks per thread");
  uint32_t v[kSlots][8];
};

template <int kThreads>
__device__ __forceinline__ void load_x_slots(const DecodeQuantArgs& q, const GemmParams& p, XSlots<kThreads>& xs) {
  const uint32_t bpr = p.K >> 4, n_blocks = p.M * bpr;
#pragma unroll
  for (int t = 0; t < XSlots<kThreads>::kSlots; ++t) {
    const uint32_t b = threadIdx.x + t * kThreads;
    if (b < n_blocks) load_x_block(q, b, bpr, xs.v[t]);
  }
}

template <int kThreads, bool kDynamic>
__device__ float quantize_into_lds(const DecodeQuantArgs& q, const GemmParams& p, XSlots<kThreads>& xs,
                                   uint8_t* lds_codes, uint8_t* lds_scales, uint32_t* red) {
  constexpr int kSlots = XSlots<kThreads>::kSlots;
  const uint32_t bpr = p.K >> 4, n_blocks = p.M * bpr;
  uint32_t (&v)[kSlots][8] = xs.v;
  uint32_t m = 0;
#pragma unroll
  for (int t = 0; t < kSlots; ++t) {
    const uint32_t b = threadIdx.x + t * kThreads;
    if (kDynamic && b < n_blocks) {
      const uint32_t a = __float_as_uint(block_amax(v[t]));
      m = m > a ? m : a;                     // non-negative floats order as integers
    }
  }
  float g;
  if (kDynamic) {
    g = global_scale(__uint_as_float(wg_max_u32<kThreads>(m, red)));
    if (blockIdx.x == 0 && threadIdx.x == 0) *q.g_enc = g;
  } else {
    g = *q.g_enc;
  }
  const float gd6 = g * (1.0f / 6.0f);
  const bool out = q.codes != nullptr && blockIdx.x == 0;
  // All blocks first, then the LDS writes: a write to LDS waits for the
  // weight ring's direct-to-LDS loads issued before it (the compiler cannot
  // tell the addresses apart), so the quantization runs before that wait.
  uint32_t c[kSlots][3];
#pragma unroll
  for (int t = 0; t < kSlots; ++t) {
    const uint32_t b = threadIdx.x + t * kThreads;
    if (b < n_blocks) {
      if (g > kHugeScale)
        c[t][2] = quantize_block<true>(v[t], g, gd6, c[t][0], c[t][1]);
      else
        c[t][2] = quantize_block<false>(v[t], g, gd6, c[t][0], c[t][1]);
    }
  }
#pragma unroll
  for (int t = 0; t < kSlots; ++t) {
    const uint32_t b = threadIdx.x + t * kThreads;
    if (b < n_blocks) {
      reinterpret_cast<uint2*>(lds_codes)[b] = make_uint2(c[t][0], c[t][1]);
      lds_scales[b] = (uint8_t)c[t][2];
      if (out) {
        reinterpret_cast<uint2*>(q.codes)[b] = make_uint2(c[t][0], c[t][1]);
        q.scales[b] = (uint8_t)c[t][2];
      }
    }
  }
  lds_barrier();
  return g;
}

// Wait until at most rem * kL loads of this wave are outstanding (rem <= R;
// rem < 0 waits for all).
template <int kL, int R>
__device__ __forceinline__ void wait_rem(int rem) {
  if constexpr (R <= 0) {
    __builtin_amdgcn_s_waitcnt(lds::vmcnt_imm(0));
  } else {
    if (rem >= R)
      __builtin_amdgcn_s_waitcnt(lds::vmcnt_imm(R * kL));
    else
      wait_rem<kL, R - 1>(rem);
  }
}

template <int KS, int FM, int FN, int kStages, bool kF32Out, bool kGate, int kQuant = 0, bool kShareA = true>
__global__ __launch_bounds__(KS * 64, 2) void gemm_splitk_kernel(const uint8_t* __restrict__ a_codes,
                                                             const uint8_t* __restrict__ a_scales,
                                                             const float* __restrict__ a_g,
                                                             const uint8_t* __restrict__ w_packed,
                                                             const float* __restrict__ w_g,
                                                             void* __restrict__ y, GemmParams p,
                                                             DecodeQuantArgs q) {
  constexpr int BM = FM * 32, BN = FN * 32;
  // With the fused quantizer the activation sits in LDS; otherwise it is
  // streamed through the workgroup's shared ring (kShareA), or, for
  // activations of a few rows (whose loads are nearly all past the rows and
  // read nothing), through each wave's private ring beside the weight, with
  // no barrier in the loop.
  constexpr bool kALds = kQuant != 0;
  constexpr bool kAShared = !kALds && kShareA;
  constexpr bool kAPrivate = !kALds && !kShareA;
  static_assert(!kALds || FM == 1, "LDS-resident activation: one 32-row fragment");
  static_assert(KS == 4, "a step is one 128-byte line group (4 chunks) of every activation row");
  using L = SplitkStage<kAPrivate ? FM : 0, FN>;
  constexpr int kWOff = kAPrivate ? FM : 0;                  // first weight slot of a private stage
  using AG = SplitkAGroup<FM>;
  constexpr int kFrags = FM + FN;
  constexpr int kScaleA = L::kScaleA, kScaleB = L::kScaleB, kStageBytes = L::kBytes;
  constexpr int kLw = L::kLoads;                             // private-ring DMA loads per step and wave
  constexpr int kLa = kAShared ? AG::kLoadsPerWave : 0;      // activation DMA loads per step and wave
  constexpr int kLoads = kLw + kLa;
  constexpr int kWaitFirst = lds::vmcnt_imm((kStages - 1) * kLoads);
  static_assert(kStages >= 2 && kStages <= 4 && (kStages - 1) * kLoads + kLw < 64, "ring depth, memory counter range");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  // The wave index is uniform: taking it through readfirstlane keeps the
  // chunk index, buffer descriptors and LDS addresses in scalar registers.
  const uint32_t lane = threadIdx.x & 63, wave = wave_index();
  const uint32_t r = lane & 31, h = lane >> 5;
  uint32_t tm, tn;
  tile_of<8>(p, tm, tn);
  const uint32_t m0 = tm * BM, n0 = tn * BN;
  constexpr int kRingBytes = splitk_ring_bytes<KS, FM, FN, kStages, kAShared>() +
                             (kAPrivate ? KS * kStages * (L::kBytes - SplitkStage<0, FN>::kBytes) : 0);
  uint8_t* ring = smem + wave * (kStages * kStageBytes);
  uint8_t* a_ring = smem + KS * kStages * kStageBytes;       // shared activation ring (kAShared)
  const uint32_t n_steps = (p.chunks + KS - 1) / KS;

  // Activation DMA of a step: wave w loads line-group slices q = w FM + t.
  // Codes, slice q: rows 8q .. 8q + 7 of the tile, 128 bytes each; lane l
  // takes 16-byte piece (l % 8) ^ (l / 8) ^ (q % 8) of row 8q + l / 8 and
  // lands at slot l (16 l) of the slice's 1 KB image, so that the 16 lanes
  // of one LDS read (rows r, the same piece) hit distinct banks.  Scales,
  // slice q: lane l < 32 takes dword l % 4 (chunk 4i + l % 4) of row
  // 8q + l / 4 (4 l in the slice's 260-byte slot; lanes >= 32 read zeros).
  uint32_t ac_off[AG::kSlicesPerWave], as_off[AG::kSlicesPerWave];
#pragma unroll
  for (int t = 0; t < AG::kSlicesPerWave; ++t) {
    const uint32_t q = wave * AG::kSlicesPerWave + t;
    const uint32_t row_c = m0 + 8 * q + (lane >> 3), piece = (lane & 7) ^ (lane >> 3) ^ (q & 7);
    ac_off[t] = (kAShared && row_c < p.M) ? row_c * (p.K >> 1) + piece * 16u : kOOB;
    const uint32_t row_s = m0 + 8 * q + (lane >> 2);
    as_off[t] = (kAShared && lane < 32 && row_s < p.M) ? row_s * (p.K >> 4) + (lane & 3) * 4u : kOOB;
  }
  // Where lane (h, r) finds its activation fragment f in a shared stage:
  // row 32 f + r, piece 2 w + h (chunk 4i + w, bytes 16 h .. 16 h + 15).
  uint32_t ar_code[FM], ar_scale[FM];
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    const uint32_t q = 4 * f + (r >> 3), rr = r & 7;
    ar_code[f] = q * 1024u + (rr * 8u + ((2 * wave + h) ^ rr ^ (q & 7))) * 16u;
    ar_scale[f] = AG::kScaleBase + q * AG::kScaleSlot + rr * 16u + wave * 4u;
  }
  // Private-ring activation: fragment f's codes, lane (h, r) the 16 bytes
  // of row r for its chunk; scale DMA of fragment pair j, lane l the scale
  // dword of row l of the pair (the missing second fragment of an odd count
  // reads zeros).
  uint32_t ap_off[FM], aps_off[L::kPairsA > 0 ? L::kPairsA : 1];
#pragma unroll
  for (int f = 0; f < FM; ++f) {
    const uint32_t row = m0 + f * 32 + r;
    ap_off[f] = row < p.M ? row * (p.K >> 1) + h * 16u : kOOB;
  }
#pragma unroll
  for (int j = 0; j < L::kPairsA; ++j) {
    const uint32_t row = m0 + 2 * j * 32 + lane;
    aps_off[j] = (2 * j + h < (uint32_t)FM && row < p.M) ? row * (p.K >> 4) : kOOB;
  }
  // Scale DMA of weight fragment pair j: lane l loads the scale dword of row
  // l % 32 of weight tile l / 32 of the pair; the missing second fragment of
  // an odd count reads zeros.
  uint32_t b_off[FN], bs_off[L::kPairsB];
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
  const __amdgpu_buffer_rsrc_t ra = rsrc(a_codes, p.a_code_bytes);
  const __amdgpu_buffer_rsrc_t rs = rsrc(a_scales, p.a_scale_bytes);
  const __amdgpu_buffer_rsrc_t rb = rsrc(w_packed, p.w_scale_offset);
  const __amdgpu_buffer_rsrc_t rbs = rsrc(w_scales, w_scale_bytes);
  // DMA of step i into stage i % kStages: this wave's share of the
  // activation line group, and the weight fragments of its chunk 4i + w.
  // (Loads of chunks past the end of K -- prologue loads when K is short, a
  // wave without a chunk in the last step -- re-load the last chunk or step
  // so that every address stays inside its tensor; they are never read.)
  auto issue_a = [&](uint32_t i) {
    if constexpr (kAShared) {
      const uint32_t iq = i < n_steps ? i : n_steps - 1;
      uint8_t* st = a_ring + (i % kStages) * AG::kBytes;
#pragma unroll
      for (int t = 0; t < AG::kSlicesPerWave; ++t) {
        const uint32_t q = wave * AG::kSlicesPerWave + t;
        dma16(ra, st + q * 1024, ac_off[t], iq * 128u);
        // Scales of chunks past the end of K read zeros: a wave without a
        // chunk in the last step then multiplies zeros into its sums.
        dma4(rs, st + AG::kScaleBase + q * AG::kScaleSlot, 4 * iq + (lane & 3) < p.chunks ? as_off[t] : kOOB,
             iq * 16u);
      }
    }
  };
  auto issue_w = [&](uint32_t i) {
    const uint32_t kc = wave + KS * i;
    const uint32_t kq = kc < p.chunks ? kc : p.chunks - 1;
    uint8_t* st = ring + (i % kStages) * kStageBytes;
    if constexpr (kAPrivate) {
#pragma unroll
      for (int f = 0; f < FM; ++f) dma16(ra, st + f * 1024, ap_off[f], kq * 32u);
#pragma unroll
      for (int j = 0; j < L::kPairsA; ++j) dma4(rs, st + kScaleA + j * 256, aps_off[j], kq * 4u);
    }
#pragma unroll
    for (int f = 0; f < FN; ++f) dma16(rb, st + (kWOff + f) * 1024, b_off[f], kq * 1024u);
#pragma unroll
    for (int j = 0; j < L::kPairsB; ++j) dma4(rbs, st + kScaleB + j * 256, bs_off[j], kq * 128u);
  };

  struct Regs {
    int4v c[kFrags];
    uint32_t s[kFrags];
  };
  // LDS-resident activation (fused quantizer): codes [M][K/2], then scales
  // [M][K/16], in a static array apart from the rings (so that its writes
  // need not wait for the ring's direct-to-LDS loads); rows >= M are zero
  // operands.
  __shared__ __attribute__((aligned(16))) uint8_t a_static[kALds ? 9 * kDecodeFuseMaxBlocks : 16];
  const uint8_t* a_lds = a_static;
  const uint8_t* as_lds = a_lds + p.M * (p.K >> 1);
  auto read_stage = [&](Regs& R, uint32_t i) {
    const uint8_t* st = ring + (i % kStages) * kStageBytes;
#pragma unroll
    for (int f = 0; f < FM; ++f) {
      if constexpr (kALds) {
        const uint32_t kc = wave + KS * i;
        const bool ok = r < p.M && kc < p.chunks;
        R.c[f] = ok ? *(const int4v*)(a_lds + r * (p.K >> 1) + kc * 32 + h * 16) : int4v{0, 0, 0, 0};
        R.s[f] = ok ? *(const uint32_t*)(as_lds + r * (p.K >> 4) + kc * 4) : 0u;
      } else if constexpr (kAPrivate) {
        R.c[f] = *(const int4v*)(st + f * 1024 + lane * 16);
        R.s[f] = *(const uint32_t*)(st + kScaleA + f * 128 + r * 4);
      } else {
        const uint8_t* as = a_ring + (i % kStages) * AG::kBytes;
        R.c[f] = *(const int4v*)(as + ar_code[f]);
        R.s[f] = *(const uint32_t*)(as + ar_scale[f]);
      }
    }
#pragma unroll
    for (int f = 0; f < FN; ++f) {
      R.c[FM + f] = *(const int4v*)(st + (kWOff + f) * 1024 + lane * 16);
      R.s[FM + f] = *(const uint32_t*)(st + kScaleB + f * 128 + r * 4);
    }
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int fa = 0; fa < FM; ++fa)
#pragma unroll
    for (int fb = 0; fb < FN; ++fb) acc[fa][fb] = floatx16{};

  // Decode + MFMA of one chunk whose raw fragments are in cur.
  auto compute = [&](const Regs& cur) {
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
  };
  // Interleave of one step: MFMAs, decode VALU, the DMA and LDS reads issued
  // after the last wait of the step.
  auto schedule = [&](auto dma_tag) {
    constexpr int kDma = decltype(dma_tag)::value;
    constexpr int kMfma = 4 * FM * FN;
    constexpr int kValu = (4 * 8 * kFrags + 2 * kFrags + kMfma - 1) / kMfma;
#pragma unroll
    for (int q = 0; q < kMfma; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, kValu, 0);                               // VALU
      if (q < kDma) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                     // VMEM (DMA)
      if (q < 2 * kFrags) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);               // LDS read
    }
  };

  float alpha[FN];
  Regs cur, nxt;
  if constexpr (!kAShared) {
    // Private rings only, no barrier: cur's stage is free once cur is in
    // registers, so it is refilled before the wait for chunk i + 1 and
    // kStages - 1 chunks stay in flight through it.  Near the end nothing
    // is refilled, and the wait for chunk i + 1 lets exactly the chunks
    // after it stay in flight (loads land in order).  With the fused
    // quantizer the weight's first stages do not depend on the activation:
    // their loads fly while the workgroup quantizes X into LDS.
    XSlots<KS * 64> xs;
    if constexpr (kALds) {
      load_x_slots<KS * 64>(q, p, xs);
      __builtin_amdgcn_sched_barrier(0);                 // X's loads first
    }
#pragma unroll
    for (int s = 0; s < kStages; ++s) issue_w(s);
    if constexpr (kALds) {
      __shared__ uint32_t red[KS];
      uint8_t* a_dst = a_static;
      const float ga = quantize_into_lds<KS * 64, kQuant == 2>(q, p, xs, a_dst, a_dst + p.M * (p.K >> 1), red);
      segment_alpha<FN>(p, ga, w_g, n0, r, alpha);
    } else {
      segment_alpha<FN>(p, *a_g, w_g, n0, r, alpha);
    }
    __builtin_amdgcn_s_waitcnt(kWaitFirst);
    const uint32_t n_mine = wave < p.chunks ? (p.chunks - 1 - wave) / KS + 1 : 0;
    read_stage(cur, 0);
    for (uint32_t i = 0; i < n_mine; ++i) {
      __builtin_amdgcn_s_waitcnt(lds::kWaitLgkm0);       // cur read from its stage
      if (i + kStages < n_mine) {
        issue_w(i + kStages);                             // refills cur's stage
        __builtin_amdgcn_s_waitcnt(lds::vmcnt_imm((kStages - 1) * kLw));   // chunk i + 1 landed
      } else {
        wait_rem<kLw, kStages - 2>((int)n_mine - 2 - (int)i);             // chunks after i + 1
      }
      read_stage(nxt, i + 1);
      compute(cur);
      schedule(std::integral_constant<int, kLw>{});
      cur = nxt;
    }
  } else {
    // Loads are issued in the order W(0), A(0), W(1), A(1), ...: W(j) (this
    // wave's weight of step j) as soon as the wave has read the stage it
    // refills, A(j) (its share of step j's activation) after the barrier
    // that says every wave has read that stage.  Every step refills (past
    // the last step with re-loads of the last chunk, into stages nobody
    // reads again), so waiting for step i + 1 always leaves in flight the
    // loads of steps i + 2 .. i + kStages - 1 and W(i + kStages).
    constexpr int kWaitStep = lds::vmcnt_imm((kStages - 2) * kLoads + kLw);
    segment_alpha<FN>(p, *a_g, w_g, n0, r, alpha);
#pragma unroll
    for (int s = 0; s < kStages; ++s) {
      issue_w(s);
      issue_a(s);
    }
    __builtin_amdgcn_s_waitcnt(kWaitFirst);
    __builtin_amdgcn_s_barrier();                          // every wave's share of step 0 landed
    read_stage(cur, 0);
    for (uint32_t i = 0; i < n_steps; ++i) {
      __builtin_amdgcn_s_waitcnt(lds::kWaitLgkm0);       // cur read from its stages
      issue_w(i + kStages);                               // this wave's weight stage is free
      __builtin_amdgcn_s_waitcnt(kWaitStep);              // this wave's loads of step i + 1 landed
      __builtin_amdgcn_s_barrier();                       // ... everyone's; every wave has read stage i
      issue_a(i + kStages);
      read_stage(nxt, i + 1);
      compute(cur);
      schedule(std::integral_constant<int, kLa>{});
      cur = nxt;
    }
  }
  // Drain this wave's DMA (prologue loads past a short K) before the ring
  // is reused for the partial sums.
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();

  constexpr int kFit = kRingBytes / (KS * 64 * 64);            // fragments whose partials fit the rings
  constexpr int kGroup = kFit < FM * FN ? kFit : FM * FN;
  static_assert(kGroup >= 1, "partial sums of one fragment fit the ring");
  splitk_epilogue<KS, FM, FN, kGroup, kF32Out, kGate>(acc, reinterpret_cast<floatx16*>(smem), p, alpha, y, m0, n0,
                                                      wave, lane);
}

template <int KS, int FM, int FN, int kStages, bool kShareA>
static hipError_t launch_splitk(const GemmOperands& o, GemmParams p, bool out_f32, bool gate, hipStream_t stream) {
  constexpr int BM = FM * 32, BN = FN * 32;
  constexpr int kLds = kShareA ? splitk_ring_bytes<KS, FM, FN, kStages, true>()
                               : KS * kStages * SplitkStage<FM, FN>::kBytes;
  static_assert(kLds >= KS * 64 * 64 && 2 * kLds <= 160 * 1024, "the reduction reuses the rings; two per CU");
  p.tiles_m = (p.M + BM - 1) / BM;
  p.tiles_n = (p.N + BN - 1) / BN;
  const dim3 grid(p.tiles_m * p.tiles_n), block(KS * 64);
#define NVFP4_SK(F32, GATE)                                                                                  \
  hipLaunchKernelGGL((gemm_splitk_kernel<KS, FM, FN, kStages, F32, GATE, 0, kShareA>), grid, block, kLds, stream, \
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
  return launch_splitk<4, 2, 3, 3, true>(o, p, out_f32, gate, stream);
}

// Activations of at most kDecodePrivateRows rows take the private rings (no
// barrier; their activation loads are a few rows of 32 bytes per chunk) and
// one weight fragment per workgroup (twice the workgroups, five per CU: 1 and
// 7 rows against the gate/up weight 30.6 -> 28.7 and 30.9 -> 29.1 us, same
// box); more rows the shared line-group ring with two weight fragments (one
// fragment would repeat the activation loads in twice the workgroups).  Each
// output column's sum runs in the same order either way.
constexpr uint32_t kDecodePrivateRows = 8;   // the kSplitkDecodeFew plan (gemm.hip) takes the same bound

hipError_t launch_splitk_decode(const GemmOperands& o, GemmParams p, bool out_f32, hipStream_t stream) {
  if (p.M <= kDecodePrivateRows) return launch_splitk<4, 1, 1, 3, false>(o, p, out_f32, false, stream);
  return launch_splitk<4, 1, 2, 3, true>(o, p, out_f32, false, stream);
}

// The fused decode path's weight ring is one stage deeper than the plain
// decode kernel's (4 instead of 3: more of the weight in flight while the
// workgroup quantizes X; one token 33.0 -> 32.6 us, same box), which still
// leaves three workgroups per CU (36 KB of ring + the 9 KB static array of
// the quantized activation each).
constexpr int kDecodeQuantStages = 4;

size_t decode_quant_lds_bytes(int64_t M, int64_t K) {
  (void)M;
  (void)K;
  return (size_t)splitk_ring_bytes<4, 1, 2, kDecodeQuantStages, false>();
}

hipError_t launch_decode_quant_gemm(const GemmOperands& o, GemmParams p, const DecodeQuantArgs& q, bool dynamic,
                                    bool out_f32, hipStream_t stream) {
  constexpr int KS = 4, FM = 1, FN = 2, kStages = kDecodeQuantStages;
  constexpr int kRing = splitk_ring_bytes<KS, FM, FN, kStages, false>();
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
