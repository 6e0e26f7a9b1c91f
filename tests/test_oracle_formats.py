"""Pins of the oracle's number formats against things other than itself:
the format's listed values, PyTorch's float8_e4m3fn decoding and casting, and
exhaustive nearest-value search."""

from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import formats as F
from tests.bruteforce import E2M1_LISTED, nearest_even


def test_e2m1_grid_is_the_listed_magnitudes():
    # E2M1 non-negative values listed for NVFP4: {0, 0.5, 1, 1.5, 2, 3, 4, 6}.
    assert F.E2M1_GRID.tolist() == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
    assert F.E2M1_MAX == 6.0


def test_e2m1_sign_bit_negates():
    for c in range(8):
        assert F.e2m1_value(c | 8) == -F.e2m1_value(c) or (c == 0 and F.e2m1_value(8) == 0.0)
    assert np.signbit(F.e2m1_value(8))


def test_e4m3_decoding_matches_torch_for_all_256_codes():
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    for code in range(256):
        ours = F.e4m3_value(code)
        if np.isnan(ref[code]):
            assert np.isnan(ours), code
        else:
            assert ours == ref[code], code


def test_e4m3_grid_extent():
    g = F.E4M3_GRID
    assert len(g) == 127
    assert g[0] == 0.0 and g[1] == 2.0 ** -9 and g[-1] == 448.0
    assert np.all(np.diff(g) > 0)


def test_e4m3_rounding_matches_torch_cast():
    rng = np.random.default_rng(1)
    vals = [np.float32(v) for v in rng.uniform(0, 464, 4000)]
    vals += [np.float32(v) for v in 2.0 ** rng.uniform(-12, 8.85, 4000)]
    mids = (F.E4M3_GRID[:-1] + F.E4M3_GRID[1:]) / 2
    for m in mids:
        m32 = np.float32(m)
        vals += [m32, np.nextafter(m32, np.float32(0)), np.nextafter(m32, np.float32(1e9))]
    vals = np.array([v for v in vals if v <= 464], dtype=np.float32)
    ours = F.E4M3_GRID[F.rne_index_sorted(vals.astype(np.float64), 1.0, F.E4M3_GRID)]
    ref = torch.from_numpy(vals).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_e4m3_saturates_above_448():
    vals = np.array([448.0, 460.0, 480.0, 1e6, 3e38])
    assert np.all(F.E4M3_GRID[F.rne_index_sorted(vals, 1.0, F.E4M3_GRID)] == 448.0)


def test_e2m1_tie_table():
    # Exact midpoints between neighbouring E2M1 values round to the even code:
    # 0.25->0, 0.75->1, 1.25->1, 1.75->2, 2.5->2, 3.5->4, 5->4; beyond 6 saturates.
    t = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 6.5, 100.0])
    expect = [0.0, 1.0, 1.0, 2.0, 2.0, 4.0, 4.0, 6.0, 6.0]
    assert F.E2M1_GRID[F.rne_index(t, 1.0, F.E2M1_GRID)].tolist() == expect


def test_rne_index_matches_exhaustive_search():
    rng = np.random.default_rng(2)
    table = list(enumerate(E2M1_LISTED))
    for _ in range(3000):
        den = float(F.E4M3_GRID[rng.integers(1, 127)])
        # numerators on and near the exact thresholds as well as at random
        base = float(rng.choice([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 7.0])) * den
        num = float(rng.choice([base, np.nextafter(base, 0), np.nextafter(base, np.inf),
                                rng.uniform(0, 7) * den]))
        ours = int(F.rne_index(num, den, F.E2M1_GRID))
        ref, _ = nearest_even(Fraction(num) / Fraction(den), table)
        assert ours == ref, (num, den)


def test_sorted_and_linear_rounding_agree():
    rng = np.random.default_rng(3)
    num = np.concatenate([rng.uniform(0, 3000, 20000), 6.0 * (F.E4M3_GRID[:-1] + F.E4M3_GRID[1:]) / 2])
    a = F.rne_index_sorted(num, 6.0, F.E4M3_GRID)
    b = F.rne_index(num, 6.0, F.E4M3_GRID)
    np.testing.assert_array_equal(a, b)


def test_bf16_decode():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x8000, 0x7F7F, 0x0001], dtype=np.uint16)
    v = F.bf16_bits_to_f64(bits)
    assert v[0] == 1.0 and v[1] == -1.0 and v[2] == 0.0 and np.signbit(v[3])
    assert v[4] == float(np.float32(3.3895313892515355e38))
    assert v[5] == 2.0 ** -133
