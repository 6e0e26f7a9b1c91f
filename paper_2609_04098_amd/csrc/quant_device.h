// Device-side NVFP4 block quantization for gfx950 (used by the activation
// quantizer and the weight prepack; never by host code).
//
// Definition (paper, section 2 "NVFP4"): one E4M3 scale per 16-element block
// set to block max / 6 under the per-tensor FP32 global scale G, elements in
// E2M1.  Every rounding is one round-to-nearest-even of the exact real value:
//
//   S    = RNE_E4M3(amax_b * G / 6)       (OCP E4M3FN, saturating at 448)
//   code = sign(x) | RNE_E2M1(|x| G / S)   (saturating at 6; 0 when S = 0)
//
// How the exact decision is reached in binary32 (no wide arithmetic):
// a value u is compared with the rounding midpoints of its target format.
// All midpoints lie on a "lattice" that is cheap to round to (for E2M1,
// q = 4 v is compared with integers; for E4M3, the grid refined by one bit).
// We round an approximation of u to the nearest lattice point L (off by far
// less than half a lattice step), then get the exact sign of u - L from one
// fused multiply-add: fma(a, G, -c L) rounds the exact value a G - c L once,
// which keeps its sign and its zero-ness (a G has <= 32 significant bits, c L
// <= 11, so the only rounding is of a non-zero difference).  Moving L by one
// ulp in that direction gives a binary32 value w that lies strictly on the
// same side as u of every midpoint, and equals a midpoint exactly when u
// does; a hardware round-to-nearest-even of w then gives the exact result.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nvfp4 {

constexpr float kRange = 2688.0f;             // 6 (E2M1 max) * 448 (E4M3 max)
constexpr float kFltMax = 3.40282347e+38f;

__device__ __forceinline__ float bf16_lo(uint32_t d) { return __uint_as_float(d << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t d) { return __uint_as_float(d & 0xFFFF0000u); }

__device__ __forceinline__ int sign3(float e) {
  // -1, 0, +1 for e < 0, e == +0, e > 0 as one v_med3_i32 on the bit
  // pattern (e is never -0.0 here: an exact zero from fma is +0 under
  // round-to-nearest-even).  NaN maps to +-1.
  // (The compiler lowers min/max here to compares and selects, so the
  // instruction is written directly.)
  int r;
  asm("v_med3_i32 %0, %1, -1, 1" : "=v"(r) : "v"(__float_as_uint(e)));
  return r;
}

// max(|a|, |b|, |c|) of finite values in one v_max3_f32 (|.| as source
// modifiers; written directly because the compiler adds canonicalizing
// maxima around fmaxf).
__device__ __forceinline__ float max3_abs(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, |%1|, |%2|, |%3|" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Per-tensor global scale G = fl32(2688 / amax); 0 for amax = 0; overflow
// saturates to the largest finite binary32 value.  The division is the
// correctly rounded IEEE division (built with correctly rounded fp32 divide).
__device__ __forceinline__ float global_scale(float amax) {
  if (amax == 0.0f) return 0.0f;
  return fminf(kRange / amax, kFltMax);
}

// Max of the bf16 magnitudes of 8 packed dwords (16 elements), as a float.
__device__ __forceinline__ float block_amax(const uint32_t v[8]) {
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  u16x2 m = __builtin_bit_cast(u16x2, v[0] & 0x7FFF7FFFu);
#pragma unroll
  for (int i = 1; i < 8; ++i)
    m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, v[i] & 0x7FFF7FFFu));
  uint32_t mx = m[0] > m[1] ? m[0] : m[1];
  return __uint_as_float(mx << 16);
}

// Value of an E4M3 scale code (OCP E4M3FN; the hardware conversion).
__device__ __forceinline__ float scale_value(uint32_t code) {
  return __builtin_amdgcn_cvt_f32_fp8((int)code, 0);
}

// Block scale S = RNE_E4M3(amax_b * G / 6), exactly, as its E4M3 code and
// its value, with rq4 ~ 4 / S (0 when S = 0).  gd6 is any approximation of
// G / 6 within a few ulps; ua = amax_b * gd6 approximates amax_b G / 6.
//
// Normal scales (ua >= 2^-6, every block but nearly-empty ones): the lattice
// of E4M3 values and midpoints is the multiples of 2^(e-4) in binade
// [2^e, 2^(e+1)); the nudged lattice point w is rounded by keeping 3
// significand bits, saturating at 448 (code 126).  (w can fall just below
// 2^-6 only when the exact value does; it then rounds to code 8 = 2^-6,
// as it must.)
// Subnormal range (ua < 2^-6): the lattice is the multiples of 2^-10 and the
// code is rint(w * 2^9) (up to 8 = 2^-6).  The branch is rarely taken: when
// no lane of a wave takes it, it costs nothing.
struct BlockScale {
  uint32_t code;
  float s;      // S, exact
  float rq4;    // ~ 4 / S (0 when S = 0)
};

// kBranch = false evaluates both ranges and selects (no branch: for callers
// whose register budget is tight, where the branch's extra live values
// would spill); the results are identical.
template <bool kBranch = true>
__device__ __forceinline__ BlockScale block_scale(float amax_b, float g, float gd6) {
  const float ua = amax_b * gd6;
  BlockScale r;
  if (!kBranch) {
    const float l_norm = __uint_as_float((__float_as_uint(ua) + 0x40000u) & 0xFFF80000u);
    const float l_sub = __builtin_rintf(ua * 1024.0f) * 0x1p-10f;
    const float l = ua >= 0x1p-6f ? l_norm : l_sub;
    const int sg = sign3(__builtin_fmaf(amax_b, g, -6.0f * l));
    const float w = __uint_as_float(__float_as_uint(l) + (uint32_t)sg);
    const uint32_t code_sub = (uint32_t)__builtin_rintf(w * 512.0f);
    const uint32_t b = __float_as_uint(w);
    uint32_t code_norm = ((b + 0x7FFFFu + ((b >> 20) & 1u)) >> 20) - 960u;
    code_norm = code_norm < 126u ? code_norm : 126u;
    r.code = w < 0x1p-6f ? code_sub : code_norm;
    r.s = scale_value(r.code);
    r.rq4 = r.s > 0.0f ? 4.0f * __builtin_amdgcn_rcpf(r.s) : 0.0f;
    return r;
  }
  if (ua >= 0x1p-6f) {
    const float l = __uint_as_float((__float_as_uint(ua) + 0x40000u) & 0xFFF80000u);
    const int sg = sign3(__builtin_fmaf(amax_b, g, -6.0f * l));    // sign(amax_b G - 6 L)
    const uint32_t b = __float_as_uint(l) + (uint32_t)sg;
    const uint32_t code = ((b + 0x7FFFFu + ((b >> 20) & 1u)) >> 20) - 960u;
    r.code = code < 126u ? code : 126u;
    r.s = scale_value(r.code);
    r.rq4 = 4.0f * __builtin_amdgcn_rcpf(r.s);
  } else {
    const float l = __builtin_rintf(ua * 1024.0f) * 0x1p-10f;
    const int sg = sign3(__builtin_fmaf(amax_b, g, -6.0f * l));
    const float w = __uint_as_float(__float_as_uint(l) + (uint32_t)sg);
    r.code = (uint32_t)__builtin_rintf(w * 512.0f);
    r.s = scale_value(r.code);
    r.rq4 = r.s > 0.0f ? 4.0f * __builtin_amdgcn_rcpf(r.s) : 0.0f;
  }
  return r;
}

// E4M3 code of RNE_E4M3(amax_b * G / 6), exactly (see block_scale).
__device__ __forceinline__ uint32_t scale_code(float amax_b, float g, float gd6) {
  return block_scale(amax_b, g, gd6).code;
}

struct ElemConsts {
  float g;      // G
  float rq4;    // ~ 4 / S            (0 when S = 0)
  float grq;    // ~ G / (S / 4)      (0 when S = 0; may overflow when G is huge)
  float sq;     // S / 4, exact
};

// G above this bound can make G * 4 / S overflow; such tensors (amax below
// about 2^-89) take the two-multiply path.  The choice is per tensor, so it
// is uniform across a launch.
constexpr float kHugeScale = 0x1p100f;

__device__ __forceinline__ ElemConsts elem_consts(float g, const BlockScale& bs) {
  ElemConsts c;
  c.g = g;
  c.sq = bs.s * 0.25f;
  c.rq4 = bs.rq4;
  c.grq = g * c.rq4;
  return c;
}

// Binary32 value w such that RNE_E2M1(w / 4) equals sign(x) RNE_E2M1(|x| G / S)
// exactly (see the header comment).  q = 4 x G / S keeps the sign of x;
// n = rint(q) is the only integer that can lie between q and its
// approximation, and the thresholds 1, 3, 5, 7, 10, 14, 20 (four times the
// E2M1 midpoints) are integers.  e = |x| G - |n| S / 4, rounded once by the
// fma (abs/neg are free source modifiers), has the exact sign of |q| - |n|;
// adding that sign to the bit pattern of n moves |n| by one ulp towards |q|
// (for n = +-0, e >= 0).  The sign of x rides along in n, including -0.0.
// Beyond the last midpoint (|q| > 20) every value saturates to 6, so a large
// |q| needs no care: n S / 4 stays exact up to |n| = 2^20, and an infinite
// q (an input far beyond a calibrated static scale) gives e = -inf and
// w = +-FLT_MAX, which the conversion saturates.  kHuge: q formed as
// (x G) (4 / S), which cannot overflow when G is near FLT_MAX.
template <bool kHuge>
__device__ __forceinline__ float e2m1_arg(float x, const ElemConsts& c) {
  float q = kHuge ? (x * c.g) * c.rq4 : x * c.grq;
  float n = __builtin_rintf(q);
  float t = n * c.sq;                                          // exact
  int s = sign3(__builtin_fmaf(__builtin_fabsf(x), c.g, -__builtin_fabsf(t)));
  return __uint_as_float(__float_as_uint(n) + (uint32_t)s);
}

// Packed codes of 8 elements (binary32 values of 8 consecutive bf16
// elements); element 2j goes to the low nibble of byte j.  The conversion
// divides by 2^exponent(4.0) = 4 and rounds to nearest even with saturation.
template <bool kHuge>
__device__ __forceinline__ uint32_t encode8(const float* f, const ElemConsts& k) {
  uint32_t r = 0u;
  r = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(r, e2m1_arg<kHuge>(f[0], k), e2m1_arg<kHuge>(f[1], k), 4.0f, 0);
  r = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(r, e2m1_arg<kHuge>(f[2], k), e2m1_arg<kHuge>(f[3], k), 4.0f, 1);
  r = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(r, e2m1_arg<kHuge>(f[4], k), e2m1_arg<kHuge>(f[5], k), 4.0f, 2);
  r = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(r, e2m1_arg<kHuge>(f[6], k), e2m1_arg<kHuge>(f[7], k), 4.0f, 3);
  return r;
}

// Quantize one block: 8 dwords of bf16 pairs -> 2 dwords of packed codes;
// returns the E4M3 scale code.  The block maximum is taken on the widened
// values (|.| is a free source modifier of the three-input maximum); it is
// exact, bf16 values being binary32 values, subnormals included.
template <bool kHuge, bool kBranch = true>
__device__ __forceinline__ uint32_t quantize_block(const uint32_t v[8], float g, float gd6,
                                                   uint32_t& c0, uint32_t& c1) {
  float f[16];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    f[2 * i] = bf16_lo(v[i]);
    f[2 * i + 1] = bf16_hi(v[i]);
  }
  float amax_b = max3_abs(f[0], f[1], f[2]);
#pragma unroll
  for (int i = 3; i < 15; i += 2) amax_b = max3_abs(amax_b, f[i], f[i + 1]);
  amax_b = max3_abs(amax_b, f[15], f[15]);
  const BlockScale bs = block_scale<kBranch>(amax_b, g, gd6);
  const ElemConsts k = elem_consts(g, bs);
  c0 = encode8<kHuge>(f, k);
  c1 = encode8<kHuge>(f + 8, k);
  return bs.code;
}

}  // namespace nvfp4
