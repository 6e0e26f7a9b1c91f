"""Pins of the GDN gate oracle (paper, Eq. 1): special values, ranges,
symmetry and monotonicity that a sign, order or argument mistake would break.
"""

import math

import numpy as np

from oracle import gates as OGa


def test_special_values():
    assert OGa.sigmoid(0.0) == 0.5
    assert OGa.softplus(0.0) == math.log(2.0)
    # A_log = 0, a + dt_bias = 0: alpha = exp(-ln 2) = 1/2.
    out = OGa.gdn_gates(np.array([[0.0, 0.7]]), [0.0], [-0.7])
    assert out[0, 0] == 0.5
    assert abs(out[0, 1] - 0.5) < 1e-15


def test_ranges_symmetry_monotonicity():
    rng = np.random.default_rng(1)
    h = 8
    a_log = rng.uniform(-2, 2, h)
    dt = rng.uniform(-3, 3, h)
    y = rng.standard_normal((200, 2 * h)) * 10
    out = OGa.gdn_gates(y, a_log, dt)
    assert np.all((out > 0) & (out < 1))
    b = y[:, :h]
    np.testing.assert_allclose(OGa.sigmoid(-b), 1 - OGa.sigmoid(b), rtol=0, atol=1e-15)
    # beta increases with b; alpha decreases with a (a larger a means more decay).
    ys = np.sort(y, axis=0)
    o2 = OGa.gdn_gates(ys, a_log, dt)
    assert np.all(np.diff(o2[:, :h], axis=0) >= 0)
    assert np.all(np.diff(o2[:, h:], axis=0) <= 0)
    # Larger A_log (faster decay) gives smaller alpha for the same input.
    o3 = OGa.gdn_gates(y, a_log + 1.0, dt)
    assert np.all(o3[:, h:] <= out[:, h:])
    np.testing.assert_array_equal(o3[:, :h], out[:, :h])


def test_log_alpha_is_minus_exp_alog_times_softplus():
    """log(alpha) = g exactly as written, checked against the textbook
    softplus log(1 + e^x) where that form is accurate."""
    rng = np.random.default_rng(2)
    h = 4
    a_log = rng.uniform(-1, 1, h)
    dt = rng.uniform(-1, 1, h)
    y = rng.uniform(-5, 5, (50, 2 * h))
    out = OGa.gdn_gates(y, a_log, dt)
    g = -np.exp(a_log)[None, :] * np.log1p(np.exp(y[:, h:] + dt[None, :]))
    np.testing.assert_allclose(np.log(out[:, h:]), g, rtol=1e-12)
    np.testing.assert_allclose(out[:, :h], 1 / (1 + np.exp(-y[:, :h])), rtol=1e-14)
