"""Pins of the oracle GEMM: two independent evaluations of the same sum (exact
int64 and float64 BLAS), the dequantize-then-matmul definition, one-hot rows,
and the per-segment global-scale invariance that fixes which scale goes with
which output column."""

import numpy as np

from oracle import gemm as G
from oracle import quant as Q
from paper_2609_04098_amd import synth


def bits_of(vals):
    return synth.f64_to_bf16_bits(np.asarray(vals, dtype=np.float64))


def _problem(rng, m=24, k=64, segs=(16, 8, 24), outlier=True):
    x = rng.standard_normal((m, k))
    if outlier:
        x[:, 5] *= 120.0
    n = sum(segs)
    offs = [0] + list(np.cumsum(segs))
    w = np.concatenate([rng.standard_normal((s, k)) * sd
                        for s, sd in zip(segs, [0.02, 0.05, 0.011, 0.3][:len(segs)])])
    ap, as_, ga = Q.quantize_tensor(bits_of(x))
    wp, ws, gw = Q.quantize_segments(bits_of(w), offs)
    return ap, as_, ga, wp, ws, gw, offs, n


def test_exact_int64_equals_f64_blas():
    rng = np.random.default_rng(20)
    for _ in range(5):
        ap, as_, ga, wp, ws, gw, offs, _ = _problem(rng)
        y1 = G.gemm_exact(ap, as_, ga, wp, ws, gw, offs)
        y2 = G.gemm_f64(ap, as_, ga, wp, ws, gw, offs)
        r = G.abs_bound(ap, as_, ga, wp, ws, gw, offs)
        assert np.all(np.abs(y1 - y2) <= 1e-13 * r + 1e-300)


def test_matches_dequantize_then_matmul():
    rng = np.random.default_rng(21)
    ap, as_, ga, wp, ws, gw, offs, n = _problem(rng)
    xa = Q.dequantize(ap, as_, ga)
    wd = np.concatenate([Q.dequantize(wp[a:b], ws[a:b], gw[s])
                         for s, (a, b) in enumerate(zip(offs, offs[1:]))])
    y = G.gemm_f64(ap, as_, ga, wp, ws, gw, offs)
    r = G.abs_bound(ap, as_, ga, wp, ws, gw, offs)
    assert np.all(np.abs(y - xa @ wd.T) <= 1e-13 * r)


def test_one_hot_rows_select_dequantized_weight_columns():
    rng = np.random.default_rng(22)
    k = 64
    x = np.zeros((k, k))
    np.fill_diagonal(x, 2.0)                      # row m is 2 * e_m: exact in NVFP4
    w = rng.standard_normal((40, k)) * 0.02
    offs = [0, 24, 40]
    ap, as_, ga = Q.quantize_tensor(bits_of(x))
    wp, ws, gw = Q.quantize_segments(bits_of(w), offs)
    y = G.gemm_exact(ap, as_, ga, wp, ws, gw, offs)
    wd = np.concatenate([Q.dequantize(wp[a:b], ws[a:b], gw[s])
                         for s, (a, b) in enumerate(zip(offs, offs[1:]))])
    assert np.allclose(Q.dequantize(ap, as_, ga), x)
    np.testing.assert_allclose(y, 2.0 * wd.T, rtol=1e-15, atol=0)


def test_segment_scale_goes_with_its_own_columns():
    # Multiplying segment s of W by 2^j multiplies its amax by 2^j, so its
    # global scale becomes exactly G_s * 2^-j while codes and block scales stay
    # the same; Y must then change by exactly 2^j on segment s's columns only.
    rng = np.random.default_rng(23)
    m, k, segs = 16, 96, (8, 16, 8)
    offs = [0] + list(np.cumsum(segs))
    x = rng.standard_normal((m, k))
    w = rng.standard_normal((sum(segs), k)) * 0.03
    ap, as_, ga = Q.quantize_tensor(bits_of(x))
    wp, ws, gw = Q.quantize_segments(bits_of(w), offs)
    y = G.gemm_exact(ap, as_, ga, wp, ws, gw, offs)
    for s, j in [(0, 3), (1, -5), (2, 7)]:
        w2 = w.copy()
        w2[offs[s]:offs[s + 1]] *= 2.0 ** j
        wp2, ws2, gw2 = Q.quantize_segments(bits_of(w2), offs)
        np.testing.assert_array_equal(wp2, wp)
        np.testing.assert_array_equal(ws2, ws)
        assert gw2[s] == np.float32(gw[s] * 2.0 ** -j)
        y2 = G.gemm_exact(ap, as_, ga, wp2, ws2, gw2, offs)
        expect = y.copy()
        expect[:, offs[s]:offs[s + 1]] *= 2.0 ** j
        np.testing.assert_array_equal(y2, expect)


def test_zero_activation_gives_zero_output():
    rng = np.random.default_rng(24)
    x = np.zeros((4, 32))
    w = rng.standard_normal((8, 32))
    ap, as_, ga = Q.quantize_tensor(bits_of(x))
    wp, ws, gw = Q.quantize_segments(bits_of(w), [0, 8])
    assert ga == 0.0
    assert np.all(G.gemm_exact(ap, as_, ga, wp, ws, gw, [0, 8]) == 0.0)
    assert np.all(G.gemm_f64(ap, as_, ga, wp, ws, gw, [0, 8]) == 0.0)


def test_abs_bound_dominates():
    rng = np.random.default_rng(25)
    ap, as_, ga, wp, ws, gw, offs, _ = _problem(rng)
    y = G.gemm_f64(ap, as_, ga, wp, ws, gw, offs)
    r = G.abs_bound(ap, as_, ga, wp, ws, gw, offs)
    assert np.all(np.abs(y) <= r * (1 + 1e-12))


def test_abs_bound_equals_y_for_nonnegative_operands():
    # With every dequantized product >= 0 the sum of |a_k w_k| is the sum
    # itself, so R must equal Y (segment scales included) on every element.
    rng = np.random.default_rng(26)
    m, k, segs = 20, 128, (8, 24, 16)
    offs = [0] + list(np.cumsum(segs))
    x = np.abs(rng.standard_normal((m, k)))
    x[:, 9] *= 150.0
    w = np.concatenate([np.abs(rng.standard_normal((s, k))) * sd for s, sd in zip(segs, (0.02, 0.5, 3e-3))])
    ap, as_, ga = Q.quantize_tensor(bits_of(x))
    wp, ws, gw = Q.quantize_segments(bits_of(w), offs)
    y = G.gemm_exact(ap, as_, ga, wp, ws, gw, offs)
    r = G.abs_bound(ap, as_, ga, wp, ws, gw, offs)
    assert np.all(y > 0)
    np.testing.assert_allclose(r, y, rtol=1e-14, atol=0)


def test_abs_bound_of_one_hot_rows():
    # Row m of X holds one non-zero value, at position k_m; then
    # R[m, n] = |x_hat[m, k_m]| * |w_hat[n, k_m]|, with x_hat and w_hat the
    # dequantized tensors (each divided by its own global scale).
    rng = np.random.default_rng(27)
    k, segs = 96, (16, 8, 40)
    offs = [0] + list(np.cumsum(segs))
    pos = rng.integers(0, k, 48)
    x = np.zeros((48, k))
    x[np.arange(48), pos] = rng.choice([-3.0, -0.5, 1.0, 6.0, 2.0], 48)
    w = np.concatenate([rng.standard_normal((s, k)) * sd for s, sd in zip(segs, (0.02, 7.0, 1e-3))])
    ap, as_, ga = Q.quantize_tensor(bits_of(x))
    wp, ws, gw = Q.quantize_segments(bits_of(w), offs)
    xh = Q.dequantize(ap, as_, ga)
    wh = np.concatenate([Q.dequantize(wp[a:b], ws[a:b], gw[s]) for s, (a, b) in enumerate(zip(offs, offs[1:]))])
    expect = np.abs(xh[np.arange(48), pos])[:, None] * np.abs(wh[:, pos]).T
    r = G.abs_bound(ap, as_, ga, wp, ws, gw, offs)
    np.testing.assert_allclose(r, expect, rtol=1e-14, atol=0)
    assert np.mean(r[:, offs[1]:offs[2]] > 0) > 0.8


def test_abs_bound_ignores_signs_and_scales_with_its_segment():
    # Flipping the sign bit of whole rows of X or W leaves R unchanged (Y
    # changes sign there); scaling segment s of W by 2^j scales only that
    # segment's columns of R by 2^j.
    rng = np.random.default_rng(28)
    ap, as_, ga, wp, ws, gw, offs, n = _problem(rng)
    r = G.abs_bound(ap, as_, ga, wp, ws, gw, offs)
    y = G.gemm_exact(ap, as_, ga, wp, ws, gw, offs)
    flip_a = np.zeros(ap.shape[0], dtype=bool)
    flip_a[::3] = True
    flip_w = np.zeros(n, dtype=bool)
    flip_w[1::2] = True
    ap2, wp2 = ap.copy(), wp.copy()
    ap2[flip_a] ^= 0x88
    wp2[flip_w] ^= 0x88
    np.testing.assert_array_equal(G.abs_bound(ap2, as_, ga, wp2, ws, gw, offs), r)
    sgn = np.where(flip_a, -1.0, 1.0)[:, None] * np.where(flip_w, -1.0, 1.0)[None, :]
    np.testing.assert_array_equal(G.gemm_exact(ap2, as_, ga, wp2, ws, gw, offs), sgn * y)
    for s, j in [(0, 4), (2, -6)]:
        gw2 = list(gw)
        gw2[s] = np.float32(gw[s] * 2.0 ** -j)
        r2 = G.abs_bound(ap, as_, ga, wp, ws, gw2, offs)
        expect = r.copy()
        expect[:, offs[s]:offs[s + 1]] *= 2.0 ** j
        np.testing.assert_allclose(r2, expect, rtol=1e-15, atol=0)
