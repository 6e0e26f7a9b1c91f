// Private layout of a prepacked NVFP4 weight, shared by the prepack kernels
// and the GEMM.
//
// W has N rows (GEMM output columns) and K columns (reduction).  N is padded
// to Np = 32 * ceil(N/32) and K to Kp = 64 * ceil(K/64); padding holds zero
// codes and zero scales.  The GEMM reads W as the B operand of
// v_mfma_f32_32x32x16_f16, one 32-column tile at a time.  In a 64-wide chunk
// of K, lane l = 32 h + r of the wave handles output column r of the tile and
// the 32 reduction indices [32 h, 32 h + 32) of the chunk; at MFMA step j
// (0..3) it supplies elements [32 h + 8 j, 32 h + 8 j + 8), which belong to
// block 4 kc + 2 h + j/2.  The same index map is used for the activation, so
// the GEMM sum is unchanged.
//
//   codes:  [Np/32][Kp/64][64 lanes][16 bytes]; lane (h, r) of tile nt,
//           chunk kc holds the canonical code bytes [kc*32 + 16 h, +16) of
//           row 32 nt + r, i.e. blocks 4 kc + 2 h (bytes 0..7) and
//           4 kc + 2 h + 1 (bytes 8..15).  One wave-wide 16-byte load per
//           tile and chunk, fully contiguous (1 KB).
//   scales: at byte offset Np*Kp/2: [Np/32][Kp/64][32 rows][4 bytes]; the
//           4 bytes of row r in tile nt, chunk kc are the E4M3 scales of
//           blocks 4 kc .. 4 kc + 3 of row 32 nt + r (128 contiguous bytes
//           per tile and chunk; lanes r and 32 + r read the same dword).
#pragma once

#include <stdint.h>

namespace nvfp4 {

struct PackedDims {
  int64_t np, kp;          // padded N, padded K
  int64_t kc;              // chunks of 64 along K
  int64_t scale_offset;    // byte offset of the scale region
  int64_t bytes;           // total bytes
};

inline PackedDims packed_dims(int64_t n, int64_t k) {
  PackedDims d;
  d.np = (n + 31) / 32 * 32;
  d.kp = (k + 63) / 64 * 64;
  d.kc = d.kp / 64;
  d.scale_offset = d.np * d.kp / 2;
  d.bytes = d.scale_offset + d.np * d.kp / 16;
  return d;
}

// Byte offset of the 8 code bytes of block kb of row n.
__host__ __device__ inline uint32_t packed_code_offset(uint32_t n, uint32_t kb, uint32_t kc_count) {
  uint32_t nt = n >> 5, r = n & 31, kc = kb >> 2, h = (kb >> 1) & 1, sub = kb & 1;
  return ((nt * kc_count + kc) * 64u + h * 32u + r) * 16u + sub * 8u;
}

// Byte offset (from the start of the scale region) of the scale of block kb
// of row n.
__host__ __device__ inline uint32_t packed_scale_offset(uint32_t n, uint32_t kb, uint32_t kc_count) {
  uint32_t nt = n >> 5, r = n & 31, kc = kb >> 2, u = kb & 3;
  return ((nt * kc_count + kc) * 32u + r) * 4u + u;
}

}  // namespace nvfp4
