"""Dequantized NVFP4 x NVFP4 GEMM with per-segment global scales.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Y = dq(A) dq(W)^T, where A is the quantized activation (M, K) with one global
scale G_a and W is a fused weight (N, K) whose output columns fall into
segments s = 0..n_seg-1, segment s having its own global scale G_w[s] (paper,
section 6: several per-module-calibrated modules served as one GEMM; each
output segment must be scaled by its own module's scale).  Because
dq(x) = e * S / G, column n of segment s is

    Y[m, n] = (1 / (G_a * G_w[s])) * sum_k (e_a S_a)[m, k] * (e_w S_w)[n, k].

``gemm_f64`` evaluates the sum with float64 BLAS on the exact unscaled values.
``gemm_exact`` evaluates it in int64 with no rounding at all: with
a = 2 e (an integer in [-12, 12]) and b = 2^9 S (an integer up to 229376),
(e_a S_a)(e_w S_w) = 2^-20 * a_a b_a a_w b_w.
``abs_bound`` is sum_k |a_k w_k| with the same scaling; the GEMM tolerance is
stated relative to it.
"""

import numpy as np

from .quant import BLOCK, decode_unscaled, unpack_nibbles
from .formats import E2M1_GRID, E4M3_GRID


def segment_alpha(g_a, g_w_seg, seg_offsets, n):
    """Per-column epilogue factor 1 / (G_a * G_w[s]) in float64 (0 when the
    product is 0, i.e. an all-zero tensor)."""
    alpha = np.empty(n, dtype=np.float64)
    offs = [int(o) for o in seg_offsets]
    for s, (a, b) in enumerate(zip(offs, offs[1:])):
        p = float(np.float32(g_a)) * float(np.float32(g_w_seg[s]))
        alpha[a:b] = 0.0 if p == 0.0 else 1.0 / p
    return alpha


def gemm_f64(a_packed, a_scales, g_a, w_packed, w_scales, g_w_seg, seg_offsets,
             rows=None):
    """Y (float64) for all rows, or for the row indices ``rows``."""
    if rows is not None:
        a_packed, a_scales = a_packed[rows], a_scales[rows]
    a = decode_unscaled(a_packed, a_scales)
    w = decode_unscaled(w_packed, w_scales)
    alpha = segment_alpha(g_a, g_w_seg, seg_offsets, w.shape[0])
    return (a @ w.T) * alpha[None, :]


def abs_bound(a_packed, a_scales, g_a, w_packed, w_scales, g_w_seg, seg_offsets,
              rows=None):
    """R[m, n] = sum_k |dq(A)[m, k] * dq(W)[n, k]| (float64)."""
    if rows is not None:
        a_packed, a_scales = a_packed[rows], a_scales[rows]
    a = np.abs(decode_unscaled(a_packed, a_scales))
    w = np.abs(decode_unscaled(w_packed, w_scales))
    alpha = segment_alpha(g_a, g_w_seg, seg_offsets, w.shape[0])
    return (a @ w.T) * np.abs(alpha)[None, :]


def _int_operands(packed, scales):
    codes = unpack_nibbles(packed).astype(np.int64)
    rows, k = codes.shape
    two_e = (2.0 * E2M1_GRID[codes & 7]).astype(np.int64)
    two_e = np.where(codes & 8, -two_e, two_e).reshape(rows, k // BLOCK, BLOCK)
    s512 = (E4M3_GRID[scales] * 512.0).astype(np.int64)     # exact integers
    return two_e, s512


def gemm_exact(a_packed, a_scales, g_a, w_packed, w_scales, g_w_seg, seg_offsets):
    """Y with the sum formed exactly in int64 (small shapes only: it builds an
    (M, N, K/16) array).  Only the final scaling by 2^-20 * alpha rounds."""
    ea, sa = _int_operands(a_packed, a_scales)
    ew, sw = _int_operands(w_packed, w_scales)
    inner = np.einsum("mbi,nbi->mnb", ea, ew)               # per-block sums
    acc = np.einsum("mnb,mb,nb->mn", inner, sa, sw)         # |acc| < 2^63
    alpha = segment_alpha(g_a, g_w_seg, seg_offsets, ew.shape[0])
    return acc.astype(np.float64) * 2.0 ** -20 * alpha[None, :]
