"""Pins of the fused-group harmonization oracle (paper, section 6,
"Per-module calibration vs. fused-GEMM scaling").

* the shared scale: the largest-amax segment's (smallest encode-direction) G;
* the fold against an independent brute force (exact rationals, E4M3 values
  from PyTorch's float8_e4m3fn), including exact ties;
* closed forms: ratio 1 is the identity, a power-of-two ratio is exact where
  the result is on the grid, the re-rounding error of a normal scale is at
  most 2^-4 (the paper's 6.2% bound) and scales only shrink;
* the faulty fused GEMM scales segment s by exactly G_s / G_shared;
* the repaired GEMM stays within the re-rounding bound of the per-segment
  result.
"""

from fractions import Fraction

import numpy as np
import pytest

from oracle import gemm as OG
from oracle.formats import E4M3_GRID
from oracle import harmonize as OH
from oracle import quant as OQ
from paper_2609_04098_amd import synth
from tests.bruteforce import E4M3_FINITE, nearest_even

E4M3_VALUES = {code: val for code, val in E4M3_FINITE}
ALL_CODES = np.arange(127, dtype=np.uint8).reshape(1, 127)


def fold_all(g_s, g_shared):
    return OH.fold_scales(ALL_CODES, [0, 1], [g_s], g_shared)[0]


def test_shared_scale_is_smallest_positive_encode_scale():
    g = np.array([3.5, 0.0, 1.25, 7.0], dtype=np.float32)
    assert OH.shared_global_scale(g) == np.float32(1.25)
    assert OH.shared_global_scale(np.zeros(3, np.float32)) == 0.0
    assert OH.shared_global_scale(np.array([np.float32(5e-39)], np.float32)) == np.float32(5e-39)


def test_fold_with_ratio_one_is_identity():
    for g in [np.float32(1.0), np.float32(2688.0 / 7.3125), np.float32(3.0e30)]:
        np.testing.assert_array_equal(fold_all(g, g), ALL_CODES[0])


def test_fold_by_power_of_two_is_exact_on_the_grid():
    values = {v: c for c, v in E4M3_FINITE}
    for k in range(0, 12):
        out = fold_all(np.float32(2.0 ** 20), np.float32(2.0 ** (20 - k)))
        for code in range(127):
            target = E4M3_VALUES[code] / 2 ** k
            if target in values:
                assert out[code] == values[target], (k, code)


def test_fold_matches_bruteforce_random_ratios():
    rng = np.random.default_rng(11)
    for _ in range(40):
        g_s = np.float32(np.exp(rng.uniform(-20, 20)))
        ratio = rng.uniform(1 / 3.0, 1.0)
        g_sh = np.float32(g_s * ratio)
        if g_sh > g_s:
            g_sh = g_s
        out = fold_all(g_s, g_sh)
        q = Fraction(float(g_sh)) / Fraction(float(g_s))
        for code in range(127):
            want, _ = nearest_even(E4M3_VALUES[code] * q, E4M3_FINITE)
            assert out[code] == want, (float(g_s), float(g_sh), code)


def test_fold_matches_bruteforce_on_exact_ties():
    """S * G_shared / G_s lands exactly on the midpoint between two E4M3
    values: the even code wins."""
    grid = sorted(E4M3_VALUES.items(), key=lambda cv: cv[1])
    checked = 0
    for code in (0x08, 0x30, 0x38, 0x3B, 0x4F, 0x7E):
        v = E4M3_VALUES[code]
        for (c0, v0), (c1, v1) in zip(grid, grid[1:]):
            mid = (v0 + v1) / 2
            if mid > v or mid == 0:
                continue
            g_s = np.float32(float(v) * 2.0 ** 30)
            g_sh = np.float32(float(mid) * 2.0 ** 30)
            assert Fraction(float(g_sh)) / Fraction(float(g_s)) * v == mid
            out = OH.fold_scales(np.array([[code]], np.uint8), [0, 1], [g_s], g_sh)[0, 0]
            want, _ = nearest_even(mid, E4M3_FINITE)
            assert want == (c0 if c0 % 2 == 0 else c1)
            assert out == want, (code, c0, c1)
            checked += 1
    assert checked > 300


def test_fold_error_bound_and_monotone():
    """Where S * ratio is in the normal E4M3 range the folded scale is within
    2^-4 relative of it (the paper's 6.2% bound); below, within half the
    subnormal spacing, 2^-10;
    folding never increases a scale and keeps the scale order."""
    rng = np.random.default_rng(12)
    vals = np.array([float(E4M3_VALUES[c]) for c in range(127)])
    for _ in range(200):
        g_s = np.float32(np.exp(rng.uniform(-10, 10)))
        g_sh = np.float32(g_s / rng.uniform(1.0, 2.81))
        out = fold_all(g_s, g_sh)
        exact = vals * (float(g_sh) / float(g_s))
        got = vals[out.astype(np.int64)]
        normal = exact >= 2.0 ** -6
        assert np.all(np.abs(got - exact)[normal] <= 2.0 ** -4 * exact[normal] * (1 + 1e-12))
        assert np.all(np.abs(got - exact)[~normal] <= 2.0 ** -10 * (1 + 1e-12))
        assert np.all(got <= vals)
        assert np.all(np.diff(out.astype(np.int64)) >= 0)


def _fused_case(seed=5, m=48, k=256, segs=(64, 96, 32), stds=(1.0, 1.5, 0.7)):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((m, k))
    x[:, rng.choice(k, 3, replace=False)] *= 80.0
    w = np.concatenate([rng.standard_normal((n, k)) * 0.02 * s for n, s in zip(segs, stds)])
    offs = [0] + list(np.cumsum(segs))
    xp, xs, gx = OQ.quantize_tensor(synth.f64_to_bf16_bits(x))
    wp, ws, gw = OQ.quantize_segments(synth.f64_to_bf16_bits(w), offs)
    return xp, xs, gx, wp, ws, gw, offs


def test_faulty_fused_gemm_scales_each_segment_by_the_scale_ratio():
    """Serving the group with G_shared and unchanged block scales multiplies
    segment s by exactly G_s / G_shared; its relative error is
    |1 - G_s / G_shared|, of the order the paper's probe reports."""
    xp, xs, gx, wp, ws, gw, offs = _fused_case()
    g_sh = OH.shared_global_scale(gw)
    n = offs[-1]
    y_ref = OG.gemm_f64(xp, xs, gx, wp, ws, gw, offs)
    y_bad = OG.gemm_f64(xp, xs, gx, wp, ws, [g_sh], [0, n])
    errs = []
    for s, (a, b) in enumerate(zip(offs, offs[1:])):
        ratio = float(gw[s]) / float(g_sh)
        np.testing.assert_allclose(y_bad[:, a:b], y_ref[:, a:b] * ratio, rtol=1e-12, atol=0)
        rel = np.linalg.norm(y_bad[:, a:b] - y_ref[:, a:b]) / np.linalg.norm(y_ref[:, a:b])
        assert rel == pytest.approx(abs(1.0 - ratio), rel=1e-9)
        errs.append(rel)
    assert min(errs) == 0.0 and max(errs) > 0.3


def test_repaired_gemm_within_rerounding_bound():
    """After the fold the one-scale GEMM differs from the per-segment result
    only by the re-rounding of block scales:
    |Y_fix - Y_ref| <= sum_b sum_{i in b} |a_i| |e_w,i| |S'_b - S_b r_s| / G_shared."""
    xp, xs, gx, wp, ws, gw, offs = _fused_case(seed=6)
    folded, g_sh = OH.harmonize(ws, offs, gw)
    n = offs[-1]
    y_ref = OG.gemm_f64(xp, xs, gx, wp, ws, gw, offs)
    y_fix = OG.gemm_f64(xp, xs, gx, wp, folded, [g_sh], [0, n])
    a = np.abs(OQ.dequantize(xp, xs, gx))
    e_w = np.abs(OQ.decode_unscaled(wp, np.full_like(ws, 0x38)))       # E2M1 values (scale 1.0)
    ratio = np.concatenate([np.full(b - a_, float(g_sh) / float(gw[s]))
                            for s, (a_, b) in enumerate(zip(offs, offs[1:]))])
    s_err = np.abs(np.array([[float(E4M3_GRID[c]) for c in row] for row in folded])
                   - np.array([[float(E4M3_GRID[c]) for c in row] for row in ws]) * ratio[:, None])
    bound = a @ (e_w * np.repeat(s_err, 16, axis=1)).T / float(g_sh)
    assert np.all(np.abs(y_fix - y_ref) <= bound * (1 + 1e-9) + 1e-300)
    rel = np.linalg.norm(y_fix - y_ref) / np.linalg.norm(y_ref)
    assert rel < 0.05
    y_bad = OG.gemm_f64(xp, xs, gx, wp, ws, [g_sh], [0, n])
    assert rel < 0.2 * np.linalg.norm(y_bad - y_ref) / np.linalg.norm(y_ref)
