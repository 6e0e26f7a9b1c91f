"""Independent brute-force NVFP4 quantizer for tiny inputs (test helper).

It shares nothing with ``oracle/``: the E4M3 values come from PyTorch's
float8_e4m3fn decoding, the E2M1 values are the format's listed magnitudes,
and rounding is done by exhaustive nearest-value search in exact rational
arithmetic (``fractions.Fraction``), ties to the even code.  The oracle
instead counts exact threshold crossings, so the two are different
algorithms for the same definition.
"""

from fractions import Fraction

import numpy as np
import torch

E2M1_LISTED = [Fraction(0), Fraction(1, 2), Fraction(1), Fraction(3, 2),
               Fraction(2), Fraction(3), Fraction(4), Fraction(6)]


def _e4m3_from_torch():
    vals = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64)
    out = []
    for code in range(256):
        v = float(vals[code])
        if np.isfinite(v) and v >= 0 and not (code & 0x80):
            out.append((code, Fraction(v)))
    return out


E4M3_FINITE = _e4m3_from_torch()     # (code, value) for the non-negative finite codes


def nearest_even(target, table):
    """(code, value) of ``table`` nearest to ``target``; ties to even code."""
    best = None
    for code, val in table:
        d = abs(val - target)
        if best is None or d < best[0] or (d == best[0] and code % 2 == 0):
            best = (d, code, val)
    return best[1], best[2]


def bf16_to_fraction(bits):
    f = np.array([int(bits) << 16], dtype=np.uint32).view(np.float32)[0]
    return Fraction(float(f))


def f32_fraction(x):
    return Fraction(float(np.float32(x)))


def exact_f32_round(q):
    """Round a positive Fraction to the nearest binary32 (ties to even
    significand) by checking the neighbours of a float candidate."""
    cand = np.float32(float(q))
    best = None
    for c in (np.nextafter(cand, np.float32(0)), cand, np.nextafter(cand, np.float32(np.inf))):
        if not np.isfinite(c):
            continue
        d = abs(Fraction(float(c)) - q)
        even = int(np.array([c], dtype=np.float32).view(np.uint32)[0]) % 2 == 0
        if best is None or d < best[0] or (d == best[0] and even):
            best = (d, c)
    return best[1]


def brute_quantize(x_bits, g):
    """Codes (rows, K) uint8 and scale codes (rows, K/16) uint8 of a tiny
    bf16 tensor under the FP32 global scale g."""
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    rows, k = x_bits.shape
    gf = f32_fraction(g)
    codes = np.zeros((rows, k), dtype=np.uint8)
    scales = np.zeros((rows, k // 16), dtype=np.uint8)
    e2m1_table = list(enumerate(E2M1_LISTED))
    for r in range(rows):
        for b in range(k // 16):
            xs = [bf16_to_fraction(x_bits[r, 16 * b + i]) for i in range(16)]
            amax = max(abs(v) for v in xs)
            s_code, s_val = nearest_even(amax * gf / 6, E4M3_FINITE)
            scales[r, b] = s_code
            for i, v in enumerate(xs):
                neg = (int(x_bits[r, 16 * b + i]) >> 15) & 1
                if s_val == 0:
                    mag = 0
                else:
                    mag, _ = nearest_even(abs(v) * gf / s_val, e2m1_table)
                codes[r, 16 * b + i] = (neg << 3) | mag
    return codes, scales
