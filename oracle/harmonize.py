"""Global-scale harmonization of a fused weight group and the mismatch it
repairs (paper, section 6, "Per-module calibration vs. fused-GEMM scaling").

TEST INFRASTRUCTURE ONLY (see the package docstring).

Several linear modules, each quantized under its own FP32 global scale G_s,
are served as one GEMM that applies a single global scale to all of its
output columns.  The paper describes two ways of forming that GEMM:

* the faulty one: one shared global scale (the "maximum" of the constituent
  scales) is used while every block scale stays as calibrated, so segment s
  is dequantized with the wrong global scale;
* the checkpoint repair: every segment is rewritten to the shared global
  scale by folding the ratio of global scales into its E4M3 block scales,
  which re-rounds them; the E2M1 codes do not change.

Readings (the paper states neither the direction of "maximum" nor how the
fold rounds):

* Global scales are held in the encode direction, G = 2688 / amax.  The
  shared scale is that of the segment with the largest amax (the maximum of
  the decode-direction scales amax / 2688), i.e. the smallest encode-direction
  G among segments with G > 0.  The fold then only shrinks block scales
  (ratio G_shared / G_s <= 1), so no block saturates at 448, and the relative
  re-rounding error of a normal E4M3 scale is at most 2^-4 (the paper bounds
  it by 6.2%).
* Folded block scale: S' = RNE_E4M3(S * G_shared / G_s), one round to nearest
  even of the exact real value (E4M3 subnormals kept, ties to the even code).
  S * G_shared has at most 4 + 24 significant bits and every threshold
  midpoint * G_s at most 5 + 24, so float64 compares them exactly.
* A segment with G_s = 0 (all of its values zero) has only zero scales and
  keeps them; it takes no part in choosing the shared scale.  If every
  segment has G_s = 0 the shared scale is 0.
"""

import numpy as np

from .formats import E4M3_GRID, rne_index_sorted


def shared_global_scale(g_seg):
    """G_shared = min over the segments' encode-direction scales that are > 0
    (the scale of the largest-amax segment); 0 if there is none."""
    g = np.asarray(g_seg, dtype=np.float32)
    pos = g[g > 0]
    return np.float32(pos.min()) if pos.size else np.float32(0.0)


def fold_scales(scales, seg_offsets, g_seg, g_shared):
    """E4M3 codes S' = RNE_E4M3(S * G_shared / G_s) for every block scale of
    every segment s (rows seg_offsets[s] .. seg_offsets[s+1] of ``scales``)."""
    scales = np.asarray(scales, dtype=np.uint8)
    out = scales.copy()
    gs = float(np.float32(g_shared))
    offs = [int(o) for o in seg_offsets]
    for s, (a, b) in enumerate(zip(offs, offs[1:])):
        g = float(np.float32(g_seg[s]))
        if g == 0.0:
            continue
        num = E4M3_GRID[scales[a:b].astype(np.int64)] * gs
        out[a:b] = rne_index_sorted(num, g, E4M3_GRID).astype(np.uint8)
    return out


def harmonize(w_scales, seg_offsets, g_seg):
    """The checkpoint repair: (folded scales, G_shared).  The weight's codes
    are unchanged; the repaired weight is one segment with scale G_shared."""
    g_shared = shared_global_scale(g_seg)
    return fold_scales(w_scales, seg_offsets, g_seg, g_shared), g_shared
