// The prefill GEMM kernel (gemm_lds_kernel) and its launcher template; each
// launched configuration is instantiated in its own translation unit
// (gemm_lds_square.hip, gemm_lds_tall.hip; the super-stage kernel, whose
// schedule takes minutes to compile, one output type per unit:
// gemm_lds_super.hip, gemm_lds_super_f32.hip).
#pragma once

#include "gemm_common.h"

namespace nvfp4 {

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
  // BF16 epilogue staging, beyond the ring (so that no wave waits for the
  // others to leave the ring): per wave 32 output rows of its FN fragment
  // columns, rows padded by 16 bytes.
  static constexpr int kEpiPitch = FN * 32 * 2 + 16;
  static constexpr int kEpiBytes = kWaves * 32 * kEpiPitch;
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
  static_assert(kOcc * (kLdsBytes + kEpiBytes) <= 160 * 1024, "LDS per CU");
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
static_assert(LdsSquare::BM == kSquareTile && LdsSquare::BN == kSquareTile && LdsSquareSuper::BN == kSquareTile,
              "square tile of the dispatch");

// BF16 epilogue of the LDS kernel: y = RNE_bf16(acc / (G_A G_W[s])) for the
// segment s of each column.  Accumulator fragment (fa, fb) is transposed:
// lane (h, r) holds output row m0 + 32 fa + r and, in entries 4 q .. 4 q + 3,
// the adjacent columns n0 + 32 fb + 8 q + 4 h + (0..3).  A whole wave block
// (all rows < M, all columns < N, one segment) with rows starting on 16-byte
// boundaries moves through the wave's own LDS staging area 32 rows at a time:
// each lane writes 8 bytes (4 columns) of one row, then every global store
// writes 16 bytes of one row, 4 lanes covering the 32 columns of a fragment
// and 16 rows per instruction (a dword per column pair spread over 4 rows
// per instruction took 3 times as long per tile in isolation, and the
// epilogue 4.8 instead of 3.3 us per tile on mlp_gate_up).  Other blocks
// (partial, unaligned, or with a segment boundary inside the wave's columns)
// are stored element by element.  The staged stores are non-temporal when
// the output is at least as large as the MALL (p.y_stream), each
// instruction then writing 4 whole rows of the wave block (256 bytes each):
// with ordinary stores, the dirty lines of mlp_gate_up's 570 MB output were
// written back during the next step's activation amax pass (dynamic
// act-quant 47.3 -> 36.4 us in the step, the GEMM and the step 0.5-0.9%
// shorter, same box).
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
constexpr int kCachePolicyNonTemporal = 2;   // the "nt" bit of a gfx950 buffer instruction

// Fast-path test and column scale of the BF16 epilogue, taken before the K
// loop so that the scale loads stay off the epilogue's path.
struct EpiPlan {
  bool whole;     // stage the wave block through LDS with one column scale
  float alpha;    // that scale
};

__device__ __forceinline__ int segment_of(const GemmParams& p, uint32_t col) {
  int s = 0;
#pragma unroll
  for (int i = 1; i < NVFP4_SEG_TABLE - 1; ++i) s += (i < p.n_seg && col >= p.seg_off[i]) ? 1 : 0;
  return s;
}

__device__ __forceinline__ float segment_scale(const float* __restrict__ a_g, const float* __restrict__ w_g, int s) {
  const float prod = *a_g * w_g[s];
  return prod == 0.0f ? 0.0f : 1.0f / prod;
}

template <int FM, int FN>
__device__ __forceinline__ EpiPlan epi_plan(const GemmParams& p, const float* __restrict__ a_g,
                                            const float* __restrict__ w_g, const void* y, uint32_t m0, uint32_t n0) {
  const uint32_t n_last = (n0 + FN * 32u < p.N ? n0 + FN * 32u : p.N) - 1u;
  const int s0 = segment_of(p, n0);
  EpiPlan e;
  e.whole = m0 + FM * 32u <= p.M && n0 + FN * 32u <= p.N && ((p.ldy * 2u) & 15u) == 0 &&
            (reinterpret_cast<uintptr_t>(y) & 15u) == 0 && s0 == segment_of(p, n_last);
  e.alpha = segment_scale(a_g, w_g, s0);
  return e;
}

template <int FM, int FN, int kPitch>
__device__ __forceinline__ void store_tile_t(const floatx16 (&acc)[FM][FN], const GemmParams& p, EpiPlan ep,
                                             const float* __restrict__ a_g, const float* __restrict__ w_g,
                                             void* __restrict__ y, uint32_t m0, uint32_t n0, uint32_t lane,
                                             uint8_t* stage) {
  constexpr uint32_t E = 2u;                      // bytes per output element
  const uint32_t r = lane & 31u, h = lane >> 5;
  if (ep.whole) {
    const float alpha = ep.alpha;
    constexpr uint32_t kPieces = 2u * E;          // 16-byte pieces per fragment row
    constexpr uint32_t kRows = 64u / kPieces;     // rows per store instruction
    const uint32_t rr = lane / kPieces, pc = lane % kPieces;
    constexpr uint32_t kLanesWide = FN * kPieces, kRowsWide = 64u / kLanesWide;   // whole wave-block rows
    const uint32_t rw = lane / kLanesWide, pw = lane % kLanesWide;
    // Non-temporal stores go through a buffer descriptor: a plain store in
    // the other branch would be merged with a non-temporal one (dropping
    // the hint).
    const __amdgpu_buffer_rsrc_t ry = rsrc(y, p.M * p.ldy * E);
#pragma unroll
    for (int fa = 0; fa < FM; ++fa) {
#pragma unroll
      for (int fb = 0; fb < FN; ++fb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const floatx16& v = acc[fa][fb];
          const uint32_t lo = pack_bf16_rne(v[4 * q] * alpha, v[4 * q + 1] * alpha);
          const uint32_t hi = pack_bf16_rne(v[4 * q + 2] * alpha, v[4 * q + 3] * alpha);
          *reinterpret_cast<u32x2*>(stage + r * kPitch + (fb * 32u + q * 8u + h * 4u) * E) = u32x2{lo, hi};
        }
      // Lanes read what other lanes wrote, and the next fragment row
      // overwrites what they read: keep the LDS accesses in program order.
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      // Byte offsets in y stay below 2^32 (the API bounds M * ldy by 2^31).
      if (p.y_stream) {
        // Non-temporal: whole 128-byte lines per instruction (a row of the
        // wave block per FN * 4 lanes); 64-byte pieces wrote 1.38 times the
        // output bytes to HBM this way.
#pragma unroll
        for (uint32_t k = 0; k < 32u / kRowsWide; ++k) {
          const uint32_t row = k * kRowsWide + rw;
          const int4v v = *reinterpret_cast<const int4v*>(stage + row * kPitch + pw * 16u);
          const uint32_t off = ((m0 + fa * 32u + row) * p.ldy + n0) * E + pw * 16u;
          __builtin_amdgcn_raw_buffer_store_b128(v, ry, off, 0, kCachePolicyNonTemporal);
        }
      } else {
#pragma unroll
        for (uint32_t k = 0; k < 32u / kRows; ++k)
#pragma unroll
          for (int fb = 0; fb < FN; ++fb) {
            const uint32_t row = k * kRows + rr;
            const int4v v = *reinterpret_cast<const int4v*>(stage + row * kPitch + fb * 32u * E + pc * 16u);
            const uint32_t off = ((m0 + fa * 32u + row) * p.ldy + n0 + fb * 32u) * E + pc * 16u;
            *reinterpret_cast<int4v*>(static_cast<uint8_t*>(y) + off) = v;
          }
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
    return;
  }
#pragma unroll
  for (int fb = 0; fb < FN; ++fb)
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t col = n0 + fb * 32u + q * 8u + h * 4u + i;
        if (col >= p.N) continue;
        const float a = segment_scale(a_g, w_g, segment_of(p, col));
#pragma unroll
        for (int fa = 0; fa < FM; ++fa) {
          const uint32_t row = m0 + fa * 32u + r;
          if (row < p.M)
            static_cast<uint16_t*>(y)[(size_t)row * p.ldy + col] = f32_to_bf16_rne(acc[fa][fb][4 * q + i] * a);
        }
      }
}

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
  // K split (FP32 partial sums): workgroup 2t + part takes chunks
  // [part * chunks, (part + 1) * chunks) of tile t; the descriptors' bases
  // move to the first of them, the row strides stay those of the whole K.
  const uint32_t part = p.k_parts > 1 ? (blockIdx.x & 1u) : 0u;
  const uint32_t kc0 = part * p.chunks;
  uint32_t tm, tn;
  tile_of<C::kGroupM>(p, tm, tn, p.k_parts > 1 ? blockIdx.x >> 1 : blockIdx.x);
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

  const __amdgpu_buffer_rsrc_t ra = rsrc(a_codes + kc0 * 32u, p.a_code_bytes - kc0 * 32u);
  const __amdgpu_buffer_rsrc_t rs = rsrc(a_scales + kc0 * 4u, p.a_scale_bytes - kc0 * 4u);
  const __amdgpu_buffer_rsrc_t rb = rsrc(w_packed + kc0 * 1024u, p.w_scale_offset - kc0 * 1024u);
  const __amdgpu_buffer_rsrc_t rbs = rsrc(w_scales + kc0 * 128u, w_scale_bytes - kc0 * 128u);
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

  // BF16 output: acc[fa][fb] holds the transposed output block of fragments
  // (fa, fb) (the MFMAs take the weight fragment as their first operand),
  // for the staged epilogue.  FP32 output keeps the direct orientation and
  // per-element stores, whose 32 lanes write 128 contiguous bytes of a row
  // (the staged form measured 3% slower there, and its instantiation's
  // main loop compiled worse).
  constexpr bool kTransposed = !kF32Out;
  const uint32_t m0_wave = tm * BM + wm * FM * 32, n0_wave = p.n_off + tn * BN + wn * FN * 32;
  EpiPlan ep{};
  if constexpr (kTransposed) ep = epi_plan<FM, FN>(p, a_g, w_g, y, m0_wave, n0_wave);
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
    // Wait for chunk c + 1's DMA and for this wave's LDS reads (those of
    // stage c were issued in the previous iteration), so that after the
    // barrier the stage of chunk c may be refilled.  The MFMAs and decode of
    // the previous chunk may still sink past the barrier; they read only
    // registers.
    if constexpr (C::kSuper)
      __builtin_amdgcn_s_waitcnt((kPos == 1 || kPos == 2 ? C::kWaitSuper1 : C::kWaitSuper0) & lds::kLgkm0Mask);
    else
      __builtin_amdgcn_s_waitcnt(C::kWaitNext & lds::kLgkm0Mask);
    __builtin_amdgcn_s_barrier();
    issue(c + kStages);
    if constexpr (kIssueSuper) issue_super((c >> 2) + 1);
    read_stage(next, c + 1);
    // Square tiles: all LDS reads of chunk c + 1 go out before this chunk's
    // MFMAs.  Left to the scheduler, half of them sank to just ahead of
    // their decode at the end of the chunk, each then waited on within one
    // MFMA (mlp_gate_up 2.17 -> 2.13 ms with the fence).
    if constexpr (C::kMfma >= 64) __builtin_amdgcn_sched_barrier(0);
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
          acc[fa][fb] = kTransposed
                            ? __builtin_amdgcn_mfma_f32_32x32x16_f16(bv[u][fb], av[u][fa], acc[fa][fb], 0, 0, 0)
                            : __builtin_amdgcn_mfma_f32_32x32x16_f16(av[u][fa], bv[u][fb], acc[fa][fb], 0, 0, 0);
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
  void* yo = kF32Out ? static_cast<void*>(static_cast<float*>(y) + (size_t)part * p.part_stride) : y;
  if constexpr (kTransposed) {
    constexpr int kPitch = C::kEpiPitch;
    store_tile_t<FM, FN, kPitch>(acc, p, ep, a_g, w_g, yo, m0_wave, n0_wave, lane,
                                 smem + C::kLdsBytes + wave * 32 * kPitch);
  } else {
    store_tile<FM, FN, kF32Out>(acc, p, a_g, w_g, yo, m0_wave, n0_wave, r, h);
  }
}

// Output columns [n_begin, n_end) (n_begin a multiple of 32).
template <class C, bool kF32Out>
static hipError_t launch_lds_as(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end,
                                hipStream_t stream) {
  p.n_off = n_begin;
  p.tiles_m = (p.M + C::BM - 1) / C::BM;
  p.tiles_n = (n_end - n_begin + C::BN - 1) / C::BN;
  const dim3 grid(p.tiles_m * p.tiles_n * p.k_parts), block(C::kThreads);
  const uint32_t lds = C::kLdsBytes + (kF32Out ? 0 : C::kEpiBytes);
  hipLaunchKernelGGL((gemm_lds_kernel<C, kF32Out>), grid, block, lds, stream, o.a_codes, o.a_scales, o.a_g,
                     o.w_packed, o.w_g, o.y, p);
  return hipGetLastError();
}

template <class C>
static hipError_t launch_lds(const GemmOperands& o, GemmParams p, uint32_t n_begin, uint32_t n_end, bool out_f32,
                             hipStream_t stream) {
  return out_f32 ? launch_lds_as<C, true>(o, p, n_begin, n_end, stream)
                 : launch_lds_as<C, false>(o, p, n_begin, n_end, stream);
}

}  // namespace nvfp4
