"""Closed forms of section 2 and Table 2 for the block statistics, and sanity
bands for the synthetic inputs (bands only: the paper's numbers come from
real activations that are not available)."""

import numpy as np

from oracle import stats as S
from oracle.formats import bf16_bits_to_f64
from paper_2609_04098_amd import synth


def test_block_max_over_rms_never_exceeds_four():
    rng = np.random.default_rng(30)
    x = rng.standard_t(1.5, (256, 64))
    x[::3, :16] = 0.0
    x[1::3, 16:32] = 0.0
    x[1::3, 17] = 5.0                        # exactly one non-zero value: ratio 4
    r = S.block_max_over_rms(x)
    r = r[np.isfinite(r)]
    assert np.all(r <= 4.0 + 1e-12)
    assert np.isclose(r.max(), 4.0)


def test_one_hot_threshold_is_energy_share():
    # max/RMS > 3 over 16 values  <=>  max^2 > (9/16) * sum(x^2) = 56.25% of energy.
    rng = np.random.default_rng(31)
    x = rng.standard_t(2, (4096, 16))
    ratio = S.block_max_over_rms(x)[:, 0]
    share = (np.abs(x).max(axis=1) ** 2) / np.sum(x * x, axis=1)
    np.testing.assert_array_equal(ratio > 3.0, share > 0.5625)


def test_synthetic_inputs_fall_in_plausible_bands():
    cfg = synth.CONFIGS["gdn_qkv"]
    x = synth.make_x(cfg, rows=512)
    st = S.tensor_stats(x)
    assert 30 < st["max_over_rms"] < 300
    assert 0.02 < st["one_hot_block_share"] < 0.3
    assert 0.02 < st["rel_quant_error"] < 0.12
    w = synth.make_w(synth.CONFIGS["tiny"])
    assert 0.07 < S.tensor_stats(w)["rel_quant_error"] < 0.13
    xt = synth.make_x(synth.CONFIGS["mlp_down"], rows=64)
    stt = S.tensor_stats(xt)
    assert 0.05 < stt["rel_quant_error"] < 0.13 and stt["one_hot_block_share"] > 0.08


def test_synth_is_deterministic_and_prefix_stable():
    cfg = synth.CONFIGS["tiny"]
    a = synth.make_x(cfg)
    b = synth.make_x(cfg)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(synth.make_x(cfg, rows=10), a[:10])
    xv = bf16_bits_to_f64(a)
    assert np.abs(xv[:, 3]).mean() > 30 and np.abs(xv[:, 100]).mean() > 30
