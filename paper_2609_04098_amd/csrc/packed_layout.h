// Private layout of a prepacked NVFP4 weight, shared by the prepack kernels
// and the GEMM.
//
// W has N rows (GEMM output columns) and K columns (reduction).  N is padded
// to Np = 32 * ceil(N/32) and K to Kp = 256 * ceil(K/256); padding holds zero
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
//           4 kc + 2 h + 1 (bytes 8..15).
//   scales: at byte offset Np*Kp/2: [Np/32][Kp/256][64 lanes][8 bytes];
//           byte 2 c + u of lane (h, r) in group kg is the E4M3 scale of
//           block 16 kg + 4 c + 2 h + u of row 32 nt + r.
#pragma once

#include <stdint.h>

namespace nvfp4 {

struct PackedDims {
  int64_t np, kp;          // padded N, padded K
  int64_t kc, kg;          // chunks of 64 and groups of 256 along K
  int64_t scale_offset;    // byte offset of the scale region
  int64_t bytes;           // total bytes
};

inline PackedDims packed_dims(int64_t n, int64_t k) {
  PackedDims d;
  d.np = (n + 31) / 32 * 32;
  d.kp = (k + 255) / 256 * 256;
  d.kc = d.kp / 64;
  d.kg = d.kp / 256;
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
__host__ __device__ inline uint32_t packed_scale_offset(uint32_t n, uint32_t kb, uint32_t kg_count) {
  uint32_t nt = n >> 5, r = n & 31, kg = kb >> 4, c = (kb >> 2) & 3, h = (kb >> 1) & 1, u = kb & 1;
  return ((nt * kg_count + kg) * 64u + h * 32u + r) * 8u + c * 2u + u;
}

}  // namespace nvfp4
