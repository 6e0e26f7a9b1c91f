"""Number formats of NVFP4 (paper, section 2 "NVFP4": E2M1 values with one E4M3
scale per 16-element block and one FP32 scale per tensor).

TEST INFRASTRUCTURE ONLY (see the package docstring).

* E2M1: 1 sign, 2 exponent, 1 mantissa bit, exponent bias 1, no inf/NaN.
  Non-negative values: 0, 0.5, 1, 1.5, 2, 3, 4, 6.
* E4M3: the OCP "E4M3FN" encoding (reading: the paper writes only "E4M3";
  the NVFP4 format uses the FN variant with max 448): 1 sign, 4 exponent,
  3 mantissa bits, bias 7, subnormals, no inf, 0x7F / 0xFF are NaN.
  Scales are non-negative, so codes 0x00..0x7E (127 values) are used.
* bf16: the top 16 bits of an IEEE binary32 value.
"""

import numpy as np

E2M1_MAX = 6.0
E4M3_MAX = 448.0
# 6 * 448: the largest magnitude a block can represent before the global scale.
NVFP4_RANGE = E2M1_MAX * E4M3_MAX


def e2m1_value(code):
    """Value of a 4-bit E2M1 code (sign in bit 3, exponent in bits 2..1,
    mantissa in bit 0, bias 1)."""
    code = int(code)
    sign = (code >> 3) & 1
    exp = (code >> 1) & 3
    man = code & 1
    if exp == 0:
        mag = man * 0.5                      # subnormal: m * 2^(1-1) / 2
    else:
        mag = (1.0 + man / 2.0) * 2.0 ** (exp - 1)
    return -mag if sign else mag


def e4m3_value(code):
    """Value of an 8-bit OCP E4M3FN code; NaN for 0x7F / 0xFF."""
    code = int(code)
    sign = (code >> 7) & 1
    exp = (code >> 3) & 15
    man = code & 7
    if exp == 15 and man == 7:
        return float("nan")
    if exp == 0:
        mag = man * 2.0 ** -9                # subnormal: (m/8) * 2^(1-7)
    else:
        mag = (1.0 + man / 8.0) * 2.0 ** (exp - 7)
    return -mag if sign else mag


# Non-negative grids, indexed by code.  Consecutive codes are consecutive
# values, so "even code" is the tie-breaking rule of round-to-nearest-even.
E2M1_GRID = np.array([e2m1_value(c) for c in range(8)], dtype=np.float64)
E4M3_GRID = np.array([e4m3_value(c) for c in range(127)], dtype=np.float64)


def rne_index(num, den, grid):
    """Index of the value of ``grid`` nearest to num/den, ties to the even
    index, saturating at the last grid value (satfinite).

    The decision compares ``num`` with ``mid * den`` for every midpoint ``mid``
    between neighbouring grid values.  Callers pass ``num`` and ``den`` such
    that both products are exact in float64, so the rounding is exact.
    ``den`` may be a scalar or broadcast against ``num``; it must be > 0.
    """
    num = np.asarray(num, dtype=np.float64)
    den = np.asarray(den, dtype=np.float64)
    idx = np.zeros(np.broadcast(num, den).shape, dtype=np.int64)
    for j in range(len(grid) - 1):
        mid = (grid[j] + grid[j + 1]) / 2.0
        thr = mid * den
        tie_goes_up = (j + 1) % 2 == 0
        idx += (num > thr) | ((num == thr) & tie_goes_up)
    return idx


def rne_index_sorted(num, den, grid):
    """Same result as ``rne_index`` for a scalar ``den``, by binary search over
    the midpoints (used for the 127-value E4M3 grid)."""
    num = np.asarray(num, dtype=np.float64)
    thr = (grid[:-1] + grid[1:]) / 2.0 * float(den)
    below = np.searchsorted(thr, num, side="left")       # thresholds < num
    at_or_below = np.searchsorted(thr, num, side="right")  # thresholds <= num
    on_tie = at_or_below > below
    # On a tie num equals thr[below], the midpoint between codes below and
    # below+1; it rounds up only when below+1 is even.
    return below + (on_tie & ((below + 1) % 2 == 0))


def bf16_bits_to_f64(bits):
    """Decode raw bf16 bit patterns (uint16) to float64, exactly."""
    bits = np.asarray(bits, dtype=np.uint16)
    f32 = (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return f32.astype(np.float64)


def f64_to_bf16_bits(y):
    """Round float64 values to bf16 once (round to nearest, ties to even),
    returning the bit patterns (uint16).  bf16 keeps 8 significant bits down
    to 2^-126 and is subnormal with spacing 2^-133 below; inputs are finite
    and inside the bf16 range."""
    y = np.asarray(y, dtype=np.float64)
    mag = np.abs(y)
    m, e = np.frexp(mag)                        # mag = m * 2^e, 0.5 <= m < 1
    normal = e - 1 >= -126
    q = np.where(normal, np.rint(np.ldexp(m, 8)), np.rint(np.ldexp(mag, 133)))
    val = np.where(normal, np.ldexp(q, e - 8), np.ldexp(q, -133))
    bits = (val.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return np.where(np.signbit(y), bits | np.uint16(0x8000), bits).astype(np.uint16)
