"""NVFP4 quantization (paper, section 2 "NVFP4").

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper fixes the format: E2M1 values, one E4M3 scale per 16-element block
set to the block maximum divided by 6, and one FP32 scale per tensor.  It does
not fix the arithmetic.  This oracle takes these readings:

* Blocks are 16 consecutive elements along K (the reduction dimension) of one
  row; K must be a multiple of 16.
* Global scale, encode direction: G = fl32(2688 / amax), 2688 = 6 * 448, so
  the tensor maximum maps onto the largest E2M1 value times the largest E4M3
  scale.  amax = 0 gives G = 0.  If the quotient overflows binary32, G is the
  largest finite binary32 value.  A "static" G (a calibrated scale) may be
  given instead.
* Block scale: S = RNE_E4M3(amax_b * G / 6), saturating at 448, with
  E4M3 subnormals kept.  Decoding divides by G.
* Element code: |code| = RNE_E2M1(|x| * G / S), saturating at 6; S = 0 gives
  magnitude 0.  The sign bit of x is always copied (so -0.0 and negative values
  that round to zero give code 0x8).
* Every rounding above is a single round-to-nearest-even of the exact real
  value.  All compared quantities are exact in float64: amax_b * G and
  |x| * G have at most 8 + 24 = 32 significant bits, and every threshold
  (grid midpoint times 6 or times S) at most 7.
* Packing: byte j of a row holds code 2j in the low nibble and code 2j+1 in
  the high nibble.  Scales are stored as E4M3 codes, one byte per block.
"""

import numpy as np

from .formats import (E2M1_GRID, E4M3_GRID, NVFP4_RANGE, bf16_bits_to_f64,
                      rne_index, rne_index_sorted)

BLOCK = 16
FLT_MAX = float(np.finfo(np.float32).max)


def tensor_amax(x_bits):
    """max |x| over a bf16 tensor given as uint16 bit patterns (exact)."""
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    if x_bits.size == 0:
        return 0.0
    mag = (x_bits & np.uint16(0x7FFF)).max()   # bf16 magnitudes order as integers
    return float(bf16_bits_to_f64(np.uint16(mag)))


def global_encode_scale(amax):
    """The per-tensor FP32 scale G = fl32(2688 / amax); 0 for amax = 0.

    The quotient is formed in float64 and then rounded to binary32.  For a
    division, rounding to 53 bits and then to 24 bits gives the same result as
    one rounding to 24 bits (53 >= 2 * 24 + 2).
    """
    amax = float(amax)
    if amax == 0.0:
        return np.float32(0.0)
    with np.errstate(over="ignore"):
        g = np.float32(NVFP4_RANGE / amax)
    if not np.isfinite(g):
        g = np.float32(FLT_MAX)
    return g


def quantize_blocks(x_bits, g):
    """Quantize a (rows, K) bf16 tensor under global scale ``g``.

    Returns (codes, scale_codes): codes uint8 (rows, K) holding 4-bit E2M1
    codes, scale_codes uint8 (rows, K/16) holding E4M3 codes.
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    rows, k = x_bits.shape
    if k % BLOCK:
        raise ValueError("K must be a multiple of 16")
    g = float(np.float32(g))
    x = bf16_bits_to_f64(x_bits).reshape(rows, k // BLOCK, BLOCK)
    ax = np.abs(x)
    amax_b = ax.max(axis=2) if k else np.zeros((rows, 0))
    # Block scale: amax_b * G / 6 rounded to E4M3.  Compare amax_b * G (exact)
    # with 6 * (E4M3 midpoints) (exact).
    scale_code = rne_index_sorted(amax_b * g, 6.0, E4M3_GRID)
    s = E4M3_GRID[scale_code]                       # (rows, K/16)
    # Element magnitude: |x| * G / S rounded to E2M1.  Compare |x| * G (exact)
    # with (E2M1 midpoints) * S (exact).
    zero_scale = s == 0.0
    den = np.where(zero_scale, 1.0, s)[:, :, None]
    mag = rne_index(ax * g, den, E2M1_GRID)
    mag[np.broadcast_to(zero_scale[:, :, None], mag.shape)] = 0
    sign = np.signbit(x).astype(np.int64)
    codes = ((sign << 3) | mag).reshape(rows, k).astype(np.uint8)
    return codes, scale_code.astype(np.uint8)


def pack_nibbles(codes):
    """(rows, K) 4-bit codes -> (rows, K/2) bytes, even k in the low nibble."""
    codes = np.asarray(codes, dtype=np.uint8)
    return (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)


def unpack_nibbles(packed):
    """(rows, K/2) bytes -> (rows, K) 4-bit codes."""
    packed = np.asarray(packed, dtype=np.uint8)
    rows, half = packed.shape
    out = np.empty((rows, 2 * half), dtype=np.uint8)
    out[:, 0::2] = packed & 0x0F
    out[:, 1::2] = packed >> 4
    return out


def quantize_tensor(x_bits, g=None, row_chunk=2048):
    """Quantize one tensor (one calibration unit) to NVFP4.

    ``g`` None: dynamic mode, G from this tensor's amax.  Otherwise the given
    (static) FP32 scale.  Returns (packed_codes (rows, K/2) uint8,
    scale_codes (rows, K/16) uint8, G as np.float32).
    Rows are processed in chunks to bound memory; blocks never span rows.
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    rows, k = x_bits.shape
    g = global_encode_scale(tensor_amax(x_bits)) if g is None else np.float32(g)
    packed = np.empty((rows, k // 2), dtype=np.uint8)
    scales = np.empty((rows, k // BLOCK), dtype=np.uint8)
    for r0 in range(0, rows, row_chunk):
        r1 = min(rows, r0 + row_chunk)
        c, s = quantize_blocks(x_bits[r0:r1], g)
        packed[r0:r1] = pack_nibbles(c)
        scales[r0:r1] = s
    return packed, scales, g


def quantize_segments(w_bits, seg_offsets, g_seg=None, row_chunk=2048):
    """Quantize a fused weight W (N, K) whose row ranges
    [seg_offsets[s], seg_offsets[s+1]) are separately calibrated modules, each
    with its own FP32 global scale (paper, section 6: one global scale per
    linear module).  Returns (packed (N, K/2), scales (N, K/16), list of G)."""
    w_bits = np.asarray(w_bits, dtype=np.uint16)
    n, k = w_bits.shape
    offs = [int(o) for o in seg_offsets]
    if offs[0] != 0 or offs[-1] != n or any(b <= a for a, b in zip(offs, offs[1:])):
        raise ValueError("segment offsets must increase strictly from 0 to N")
    packed = np.empty((n, k // 2), dtype=np.uint8)
    scales = np.empty((n, k // BLOCK), dtype=np.uint8)
    gs = []
    for s, (a, b) in enumerate(zip(offs, offs[1:])):
        gstat = None if g_seg is None else g_seg[s]
        p, sc, g = quantize_tensor(w_bits[a:b], gstat, row_chunk)
        packed[a:b] = p
        scales[a:b] = sc
        gs.append(np.float32(g))
    return packed, scales, gs


def decode_unscaled(packed, scales):
    """E2M1 value times E4M3 block scale, without the global scale, as float64
    (exact: at most 6 significant bits)."""
    codes = unpack_nibbles(packed)
    rows, k = codes.shape
    mag = E2M1_GRID[codes & 7]
    val = np.where(codes & 8, -mag, mag).reshape(rows, k // BLOCK, BLOCK)
    return (val * E4M3_GRID[scales][:, :, None]).reshape(rows, k)


def dequantize(packed, scales, g):
    """x_hat = E2M1 value * E4M3 scale / G (0 when G = 0)."""
    g = float(np.float32(g))
    v = decode_unscaled(packed, scales)
    return v / g if g != 0.0 else np.zeros_like(v)
