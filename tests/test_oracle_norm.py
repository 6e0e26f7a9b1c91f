"""Pins of the RMSNorm oracle and of the float64 -> bf16 rounding it uses.

* the rounding against a brute-force nearest-value search in exact rationals
  (random values over the whole bf16 range, subnormals, exact midpoints);
* closed forms of the norm: a constant row maps to +-gamma, a one-hot row of
  length K to sqrt(K) at the hot position, scaling a row by 2^j changes
  nothing (eps = 0), and mean(y^2) = 1 for gamma = 1, eps = 0;
* where eps enters: a constant row c with eps = c^2 maps to gamma / sqrt(2),
  a one-hot row 8 e_k of length 64 with eps = 3 to 4 gamma_k, and a zero row
  with eps > 0 to zeros.
"""

from fractions import Fraction

import numpy as np

from oracle import formats as OF
from oracle import norm as ON
from paper_2609_04098_amd import synth


def bf16_value(bits):
    return Fraction(float(np.array([int(bits) << 16], dtype=np.uint32).view(np.float32)[0]))


def brute_bf16(t):
    """Nearest bf16 to the rational t (ties to the even bit pattern)."""
    sign = 0x8000 if t < 0 else 0
    a = abs(t)
    f = np.float32(float(a))
    base = int(f.view(np.uint32)) >> 16
    best = None
    for b in range(max(0, base - 2), min(0x7F7F, base + 3) + 1):
        d = abs(bf16_value(b) - a)
        if best is None or d < best[0] or (d == best[0] and b % 2 == 0):
            best = (d, b)
    return best[1] | sign


def test_f64_to_bf16_matches_bruteforce():
    rng = np.random.default_rng(3)
    vals = list(rng.standard_normal(300) * np.exp(rng.uniform(-80, 80, 300)))
    vals += list(rng.uniform(-1, 1, 100) * 2.0 ** -128)                 # bf16 subnormals
    for b in rng.integers(1, 0x7F7E, 200):                              # exact midpoints
        vals.append(float((bf16_value(b) + bf16_value(b + 1)) / 2))
        vals.append(-float((bf16_value(b) + bf16_value(b + 1)) / 2))
    vals += [0.0, -0.0, 1.0, 2.0 ** -133, 3 * 2.0 ** -134]
    got = OF.f64_to_bf16_bits(np.array(vals))
    for v, g in zip(vals, got):
        want = brute_bf16(Fraction(v)) if v != 0 else (0x8000 if np.signbit(v) else 0)
        assert int(g) == want, (v, hex(int(g)), hex(want))


def _bits(v):
    return synth.f64_to_bf16_bits(np.asarray(v, dtype=np.float64))


def test_constant_row_maps_to_gamma():
    rng = np.random.default_rng(4)
    gamma = _bits(rng.uniform(0.5, 2.0, 256))
    x = _bits(np.array([[3.25] * 256, [-0.0078125] * 256, [1e-20] * 256]))
    y = ON.rmsnorm_f64(x, gamma, 0.0)
    g = OF.bf16_bits_to_f64(gamma)
    np.testing.assert_array_equal(y, np.stack([g, -g, g]))


def test_one_hot_row():
    x = np.zeros((2, 64), dtype=np.uint16)
    x[0, 5] = _bits(7.5)
    x[1, 63] = _bits(-0.375)
    y = ON.rmsnorm_f64(x, _bits(np.ones(64)), 0.0)
    assert y[0, 5] == 8.0 and y[1, 63] == -8.0
    assert np.count_nonzero(y) == 2


def test_power_of_two_scaling_and_unit_rms():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((8, 512))
    x[:, 7] *= 100
    gamma = _bits(np.ones(512))
    y0 = ON.rmsnorm_bf16(_bits(x), gamma, 0.0)
    for j in (-20, -3, 5, 40):
        np.testing.assert_array_equal(ON.rmsnorm_bf16(_bits(x * 2.0 ** j), gamma, 0.0), y0)
    yf = ON.rmsnorm_f64(_bits(x), gamma, 0.0)
    np.testing.assert_allclose(np.mean(yf * yf, axis=1), 1.0, rtol=1e-12)


def test_eps_inside_the_square_root():
    # y = x / sqrt(mean x^2 + eps) * gamma: a constant row c with eps = c^2
    # gives c / sqrt(2 c^2) = 1 / sqrt(2) times gamma.
    rng = np.random.default_rng(6)
    gamma = _bits(rng.uniform(0.5, 2.0, 128))
    g = OF.bf16_bits_to_f64(gamma)
    for c in (0.5, 3.0, 0.0625):
        y = ON.rmsnorm_f64(_bits(np.full((2, 128), c) * np.array([[1.0], [-1.0]])), gamma, c * c)
        np.testing.assert_allclose(y[0] * np.sqrt(2.0), g, rtol=1e-15)
        np.testing.assert_allclose(y[1] * np.sqrt(2.0), -g, rtol=1e-15)


def test_eps_with_one_hot_and_zero_rows():
    # 8 e_k in a row of 64: mean x^2 = 1, so with eps = 3 the hot value maps
    # to 8 / sqrt(4) = 4 times gamma_k.  A zero row with eps > 0 maps to 0.
    rng = np.random.default_rng(7)
    gamma = _bits(rng.uniform(0.5, 2.0, 64))
    g = OF.bf16_bits_to_f64(gamma)
    x = np.zeros((3, 64), dtype=np.uint16)
    x[0, 11] = _bits(8.0)
    x[1, 0] = _bits(-8.0)
    y = ON.rmsnorm_f64(x, gamma, 3.0)
    assert y[0, 11] == 4.0 * g[11] and y[1, 0] == -4.0 * g[0]
    assert np.count_nonzero(y[:2]) == 2
    assert np.all(y[2] == 0.0) and np.all(np.isfinite(y))
