"""Pins of the oracle quantizer: exhaustive and random comparison with an
independent rational brute-force quantizer, closed forms that follow from the
format definition, the paper's outlier-localization property, error bounds,
and a hand-derived worked example."""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import formats as F
from oracle import quant as Q
from tests import bruteforce as B
from paper_2609_04098_amd import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def bits_of(vals):
    return synth.f64_to_bf16_bits(np.asarray(vals, dtype=np.float64))


# ---------------------------------------------------------------- global scale

def test_global_scale_is_exact_binary32_quotient():
    rng = np.random.default_rng(10)
    amaxes = synth.bf16_bits_to_f32(bits_of(2.0 ** rng.uniform(-30, 30, 500)))
    for a in amaxes:
        g = Q.global_encode_scale(float(a))
        assert g == B.exact_f32_round(Fraction(2688) / Fraction(float(a))), a


def test_global_scale_edges():
    assert Q.global_encode_scale(0.0) == 0.0
    tiny = float(synth.bf16_bits_to_f32(np.array([1], dtype=np.uint16))[0])   # 2^-133
    assert Q.global_encode_scale(tiny) == np.float32(np.finfo(np.float32).max)
    assert Q.global_encode_scale(2688.0) == 1.0


# ------------------------------------------------------- brute-force agreement

def _random_tiny_tensors(rng):
    shapes = [(1, 16), (3, 32), (2, 64), (4, 48)]
    for shape in shapes:
        yield rng.standard_normal(shape)
        x = rng.standard_normal(shape)
        x[:, rng.integers(0, shape[1])] *= 150.0          # an outlier channel
        yield x
        yield rng.standard_t(3, shape) * 0.5
        x = rng.standard_normal(shape) * 1e-3
        x[0, 0] = 1e4                                      # subnormal-scale blocks
        yield x
        x = rng.standard_normal(shape)
        x[:, :16] = 0.0                                    # an all-zero block
        yield x


def test_quantizer_matches_bruteforce_dynamic():
    rng = np.random.default_rng(11)
    for x in _random_tiny_tensors(rng):
        xb = bits_of(x)
        packed, scales, g = Q.quantize_tensor(xb)
        codes_ref, scales_ref = B.brute_quantize(xb, g)
        np.testing.assert_array_equal(scales, scales_ref)
        np.testing.assert_array_equal(Q.unpack_nibbles(packed), codes_ref)


def test_quantizer_matches_bruteforce_static_scales():
    rng = np.random.default_rng(12)
    for g in [1.0, 0.375, 7.0, 1e-3, 3e3]:
        for x in _random_tiny_tensors(rng):
            xb = bits_of(x)
            packed, scales, _ = Q.quantize_tensor(xb, g=np.float32(g))
            codes_ref, scales_ref = B.brute_quantize(xb, g)
            np.testing.assert_array_equal(scales, scales_ref)
            np.testing.assert_array_equal(Q.unpack_nibbles(packed), codes_ref)


def test_every_bf16_magnitude_in_a_block_against_bruteforce():
    # Fixed global scale and a fixed block max, so the block scale is fixed;
    # the other 15 positions sweep every positive bf16 value below the max.
    g = np.float32(1.0)
    amax_bits = bits_of([3.0])[0]                  # S = RNE_E4M3(3/6) = 0.5
    below = np.arange(0x3000, int(amax_bits), dtype=np.uint16)   # 2^-31 .. <3
    rows = []
    for i in range(0, len(below), 15):
        chunk = below[i:i + 15]
        row = np.full(16, amax_bits, dtype=np.uint16)
        row[1:1 + len(chunk)] = chunk
        rows.append(row)
    xb = np.stack(rows)
    codes, scales = Q.quantize_blocks(xb, g)
    codes_ref, scales_ref = B.brute_quantize(xb, g)
    np.testing.assert_array_equal(scales, scales_ref)
    np.testing.assert_array_equal(codes, codes_ref)


def test_block_scale_decision_boundaries():
    # With G = 1 every E4M3 midpoint m gives an exactly representable block max
    # 6m, an exact tie; also one bf16 step either side of it.
    g = np.float32(1.0)
    mids = (F.E4M3_GRID[:-1] + F.E4M3_GRID[1:]) / 2
    vals = []
    for m in mids:
        b = int(bits_of([6.0 * m])[0])
        if float(synth.bf16_bits_to_f32(np.array([b], np.uint16))[0]) == 6.0 * m:
            vals += [b - 1, b, b + 1]
    xb = np.zeros((len(vals), 16), dtype=np.uint16)
    xb[:, 0] = np.array(vals, dtype=np.uint16)
    codes, scales = Q.quantize_blocks(xb, g)
    codes_ref, scales_ref = B.brute_quantize(xb, g)
    np.testing.assert_array_equal(scales, scales_ref)
    np.testing.assert_array_equal(codes, codes_ref)
    assert len(vals) > 200


# --------------------------------------------------------------- closed forms

def test_dynamic_mode_amax_block_gets_largest_scale_and_code():
    # G = fl32(2688/amax) so amax * G / 6 = 448 (1 + d), |d| <= 2^-24, which
    # rounds to 448; the amax element then maps to 6 (code 7).
    rng = np.random.default_rng(13)
    for _ in range(20):
        x = rng.standard_normal((8, 64)) * 10.0 ** rng.uniform(-20, 20)
        xb = bits_of(x)
        packed, scales, g = Q.quantize_tensor(xb)
        mag = xb & 0x7FFF
        r, c = np.unravel_index(np.argmax(mag), mag.shape)
        assert scales[r, c // 16] == 0x7E
        assert Q.unpack_nibbles(packed)[r, c] & 7 == 7


def test_zero_scale_rule():
    # S = 0 exactly when amax_b * G / 6 <= 2^-10 (half the smallest subnormal
    # 2^-9; the tie rounds to the even code 0); such blocks have magnitude 0.
    g = np.float32(1.0)
    edge = 6.0 * 2.0 ** -10
    eb = int(bits_of([edge])[0])
    xb = np.zeros((4, 16), dtype=np.uint16)
    xb[:, 0] = np.array([eb, eb + 1, bits_of([edge / 2])[0], eb | 0x8000], dtype=np.uint16)
    xb[:, 1] = bits_of([-1e-30] * 4)
    codes, scales = Q.quantize_blocks(xb, g)
    assert scales[:, 0].tolist()[0] == 0 and scales[1, 0] == 1 and scales[2, 0] == 0
    assert scales[3, 0] == 0
    for r in (0, 2, 3):
        assert np.all(codes[r] & 7 == 0)
        assert codes[r, 1] == 0x8            # sign of x is copied


def test_all_zero_tensor_and_signed_zero():
    xb = np.zeros((2, 32), dtype=np.uint16)
    xb[1, 5] = 0x8000                        # -0.0
    packed, scales, g = Q.quantize_tensor(xb)
    assert g == 0.0 and np.all(scales == 0)
    codes = Q.unpack_nibbles(packed)
    assert codes[1, 5] == 0x8 and np.sum(codes != 0) == 1
    assert np.all(Q.dequantize(packed, scales, g) == 0.0)


def test_scale_is_monotone_in_block_max():
    g = np.float32(0.731)
    vals = np.sort(2.0 ** np.random.default_rng(14).uniform(-14, 12, 3000))
    xb = np.zeros((len(vals), 16), dtype=np.uint16)
    xb[:, 3] = bits_of(vals)
    _, scales = Q.quantize_blocks(xb, g)
    assert np.all(np.diff(scales[:, 0].astype(int)) >= 0)


def test_outlier_degrades_only_its_own_block():
    # Section 2 (NVFP4): with G held fixed, each block's scale and codes depend
    # on that block's 16 values alone; planting a large value in one block
    # must leave every other block's bytes as they were.
    rng = np.random.default_rng(15)
    x = rng.standard_normal((6, 128))
    g = np.float32(5.0)
    base_p, base_s, _ = Q.quantize_tensor(bits_of(x), g=g)
    x2 = x.copy()
    x2[2, 37] = 80.0
    p2, s2, _ = Q.quantize_tensor(bits_of(x2), g=g)
    c1, c2 = Q.unpack_nibbles(base_p), Q.unpack_nibbles(p2)
    changed_blocks = {(r, c // 16) for r, c in zip(*np.nonzero(c1 != c2))}
    changed_blocks |= {(r, b) for r, b in zip(*np.nonzero(base_s != s2))}
    assert changed_blocks == {(2, 2)}


def test_dequantization_error_bound():
    # For a normal block scale, |dq(x) - x| <= half the E2M1 grid step around
    # |x| G / S, times S / G; in the saturation zone (v > 6) the error is
    # (v - 6) S / G <= 0.375 S / G since v <= 6 (1 + 2^-4).
    rng = np.random.default_rng(16)
    x = rng.standard_normal((64, 256))
    x[:, rng.choice(256, 3, replace=False)] *= 120.0
    xb = bits_of(x)
    packed, scales, g = Q.quantize_tensor(xb)
    xv = F.bf16_bits_to_f64(xb)
    xq = Q.dequantize(packed, scales, g)
    s = np.repeat(F.E4M3_GRID[scales], 16, axis=1)
    normal = s >= 2.0 ** -6
    v = np.abs(xv) * float(g) / np.where(s > 0, s, 1)
    half_step = np.where(v < 2, 0.25, np.where(v < 4, 0.5, 1.0))
    bound = np.where(v > 6, v - 6, half_step) * s / float(g)
    err = np.abs(xq - xv)
    assert np.all(err[normal] <= bound[normal] * (1 + 1e-12))
    assert np.all((v[normal] <= 6) | (v[normal] - 6 <= 0.375 + 1e-12))


def test_pack_nibble_order():
    codes = np.array([[1, 2, 3, 4, 0xF, 0x8]], dtype=np.uint8)
    assert Q.pack_nibbles(codes).tolist() == [[0x21, 0x43, 0x8F]]
    np.testing.assert_array_equal(Q.unpack_nibbles(Q.pack_nibbles(codes)), codes)


def test_hand_worked_example():
    with open(os.path.join(HERE, "golden", "worked_block.json")) as f:
        ex = json.load(f)
    xb = bits_of([ex["x"]])
    packed, scales, g = Q.quantize_tensor(xb, g=np.float32(ex["g"]))
    assert scales.tolist() == [ex["scale_codes"]]
    assert Q.unpack_nibbles(packed).tolist() == [ex["codes"]]
    np.testing.assert_array_equal(Q.dequantize(packed, scales, g)[0], ex["dequant"])


def test_segments_quantize_with_their_own_scales():
    # Section 6: one FP32 global scale per module; each segment of a fused
    # weight is quantized under its own scale, given (static) or from its amax.
    rng = np.random.default_rng(17)
    offs = [0, 2, 5, 6]
    w = np.concatenate([rng.standard_normal((2, 32)) * 0.02, rng.standard_normal((3, 32)) * 0.5,
                        rng.standard_normal((1, 32)) * 3.0])
    wb = bits_of(w)
    for g_seg in (None, [np.float32(100.0), np.float32(3.0), np.float32(0.25)]):
        packed, scales, gs = Q.quantize_segments(wb, offs, g_seg)
        for s, (a, b) in enumerate(zip(offs, offs[1:])):
            if g_seg is None:
                amax = max(abs(float(v)) for v in synth.bf16_bits_to_f32(wb[a:b]).ravel())
                assert gs[s] == B.exact_f32_round(Fraction(2688) / Fraction(amax))
            else:
                assert gs[s] == g_seg[s]
            codes_ref, scales_ref = B.brute_quantize(wb[a:b], gs[s])
            np.testing.assert_array_equal(scales[a:b], scales_ref)
            np.testing.assert_array_equal(Q.unpack_nibbles(packed[a:b]), codes_ref)
