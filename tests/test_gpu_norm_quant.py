"""GPU parity of the fused RMSNorm + static-scale quantizer
(nvfp4_rmsnorm_quantize_act).

* The normalized bf16 values y agree with the oracle's (one rounding of the
  float64 RMSNorm) except where the exact value lies within the kernel's
  binary32 error of a bf16 rounding midpoint; those differ by one bf16 step.
  The window is the binary32 error bound of the kernel's operation order
  (near_tie below), about 3e-6 relative at K = 5120.
* Codes and scales are bit-exact against the oracle quantizer applied to the
  kernel's own y with the same static G, and equal to what the stand-alone
  quantizer writes for that y on the GPU.
"""

import numpy as np
import pytest
import torch

from oracle import formats as OF
from oracle import norm as ON
from oracle import quant as OQ
from paper_2609_04098_amd import linear as L
from paper_2609_04098_amd import nvfp4 as C
from paper_2609_04098_amd import synth
from tests.gpu_common import log, np_u8, to_dev_bf16

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24        # unit roundoff of binary32


def near_tie(k):
    """Relative error bound of the kernel's binary32 y before its bf16
    rounding, for rows of k elements.  Lane sums: ceil(k / 1024) blocks of 8
    v_dot2_f32_bf16 steps, each adding two exact squares (counted as two
    roundings); a 6-level butterfly: 6 more.  A sum of n positive terms with
    m roundings is within m u relative.  Then s / K and + eps (2 roundings),
    the square root (halves the relative error, adds 1/2 u), 1 / (u), x * r
    and * gamma (2 u): |dy / y| <= (m + 2) u / 2 + 3.5 u, m = 16 ceil(k / 1024)
    + 6.  (First-order bound; the second-order terms are below 1e-10.)"""
    m = 16 * (-(-k // 1024)) + 6
    return ((m + 2) / 2.0 + 3.5) * U32


def _bits(v):
    return synth.f64_to_bf16_bits(np.asarray(v, dtype=np.float64))


def _u16(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def check_y(y_bits, x_bits, gamma_bits, eps, what):
    """y from the GPU against the float64 RMSNorm rounded once to bf16."""
    yf = ON.rmsnorm_f64(x_bits, gamma_bits, eps)
    ref = OF.f64_to_bf16_bits(yf)
    bad = y_bits != ref
    n_bad = int(bad.sum())
    if n_bad:
        # Each mismatch is one bf16 step, at a value within binary32 error of
        # the midpoint between the two candidates.
        a = OF.bf16_bits_to_f64(y_bits[bad])
        b = OF.bf16_bits_to_f64(ref[bad])
        steps = np.abs(y_bits[bad].astype(np.int64) - ref[bad].astype(np.int64))
        assert np.all(steps == 1), "%s: mismatch by more than one bf16 step" % what
        mid = (a + b) / 2
        tol = near_tie(x_bits.shape[1])
        assert np.all(np.abs(yf[bad] - mid) <= tol * np.abs(yf[bad])), "%s: mismatch away from a tie" % what
    # The bound is a few 1e-6 relative and the bf16 step 2^-8: at most a few
    # values in 10^4 can sit that close to a midpoint.
    assert n_bad <= max(4, y_bits.size // 1000), "%s: %d mismatches" % (what, n_bad)
    return n_bad


def run_fused(x_bits, gamma_bits, eps, g, ldx=None, with_y=True):
    m, k = x_bits.shape
    if ldx is None:
        x = to_dev_bf16(x_bits)
    else:
        buf = np.zeros((m, ldx), dtype=np.uint16)
        buf[:, :k] = x_bits
        x = to_dev_bf16(buf)[:, :k]
    gamma = to_dev_bf16(gamma_bits)
    y = torch.empty((m, k), dtype=torch.bfloat16, device="cuda") if with_y else None
    aq = L.rmsnorm_quantize_act(x, gamma, eps, g, y=y)
    torch.cuda.synchronize()
    return aq, y


def _case(seed, m, k, outliers=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((m, k))
    if outliers:
        x[:, rng.choice(k, max(1, k // 200), replace=False)] *= rng.uniform(50, 200)
    gamma = rng.uniform(0.5, 1.5, k)
    return _bits(x), _bits(gamma)


@pytest.mark.parametrize("m,k,ldx,eps,gfac", [
    (64, 256, None, 1e-6, 1.0),        # G from the normalized tensor's amax
    (33, 80, None, 1e-5, 0.6),         # 5 blocks: the pair's second wave has none; odd M; G too small
    (8, 5120, 5184, 1e-6, 3.0),        # strided rows; G too large: many small codes
    (5, 17408, None, 0.0, 1.0),        # the MLP-down width, eps = 0
    (3000, 1040, None, 1e-6, 1.0),     # 65 blocks: one block in the pair's second wave
    (20, 8192, 8200, 1e-6, 1.0),       # the longest row held in registers (4 blocks per lane), strided
])
def test_fused_matches_oracle(m, k, ldx, eps, gfac):
    x, gamma = _case(m + k, m, k)
    g = np.float32(OQ.global_encode_scale(np.abs(ON.rmsnorm_f64(x, gamma, eps)).max()) * gfac)
    aq, y = run_fused(x, gamma, eps, g, ldx=ldx)
    y_bits = _u16(y)
    check_y(y_bits, x, gamma, eps, "%dx%d" % (m, k))
    xp, xs, _ = OQ.quantize_tensor(y_bits, g=g)
    np.testing.assert_array_equal(np_u8(aq.codes), xp)
    np.testing.assert_array_equal(np_u8(aq.scales), xs)
    # The stand-alone quantizer on the same y, static mode: the same bytes.
    aq2 = L.quantize_act(y, g=float(g))
    torch.cuda.synchronize()
    assert torch.equal(aq2.codes, aq.codes) and torch.equal(aq2.scales, aq.scales)
    # Without the optional y output the codes are the same.
    aq3, _ = run_fused(x, gamma, eps, g, ldx=ldx, with_y=False)
    assert torch.equal(aq3.codes, aq.codes) and torch.equal(aq3.scales, aq.scales)


def test_fused_zero_and_tiny_rows():
    x, gamma = _case(9, 6, 512)
    x[1] = 0
    x[3] = _bits(np.full(512, 1e-30))
    g = np.float32(100.0)
    aq, y = run_fused(x, gamma, 1e-6, g)
    y_bits = _u16(y)
    check_y(y_bits, x, gamma, 1e-6, "zero rows")
    assert np.all(y_bits[1] == 0)
    xp, xs, _ = OQ.quantize_tensor(y_bits, g=g)
    np.testing.assert_array_equal(np_u8(aq.codes), xp)
    np.testing.assert_array_equal(np_u8(aq.scales), xs)


def test_fused_huge_static_scale():
    """A static G above 2^100 takes the quantizer's two-multiply path; every
    block saturates (scale 448, codes +-6 except zeros)."""
    x, gamma = _case(10, 4, 256)
    g = np.float32(3e36)
    aq, y = run_fused(x, gamma, 1e-6, g)
    xp, xs, _ = OQ.quantize_tensor(_u16(y), g=g)
    np.testing.assert_array_equal(np_u8(aq.codes), xp)
    np.testing.assert_array_equal(np_u8(aq.scales), xs)
    assert np.all(xs == 126)


def test_fused_empty():
    gamma = to_dev_bf16(_bits(np.ones(64)))
    codes = torch.empty((0, 32), dtype=torch.uint8, device="cuda")
    scales = torch.empty((0, 4), dtype=torch.uint8, device="cuda")
    g = torch.ones(1, dtype=torch.float32, device="cuda")
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    C.nvfp4_rmsnorm_quantize_act(x, gamma, 1e-6, codes, scales, g)
    torch.cuda.synchronize()


def test_fused_full_mlp_gate_up_activation():
    """The bench activation (8192 x 5120, residual-stream statistics) with
    gamma ~ U(0.5, 1.5) and G calibrated from the normalized tensor."""
    x = synth.make_x(synth.CONFIGS["mlp_gate_up"])
    gamma = _bits(np.random.default_rng(77).uniform(0.5, 1.5, x.shape[1]))
    eps = 1e-6
    g = OQ.global_encode_scale(np.abs(ON.rmsnorm_f64(x, gamma, eps)).max())
    aq, y = run_fused(x, gamma, eps, g)
    y_bits = _u16(y)
    n_bad = check_y(y_bits, x, gamma, eps, "mlp_gate_up")
    log("fused norm: %d of %d bf16 values on a binary32 tie" % (n_bad, y_bits.size))
    xp, xs, _ = OQ.quantize_tensor(y_bits, g=g)
    np.testing.assert_array_equal(np_u8(aq.codes), xp)
    np.testing.assert_array_equal(np_u8(aq.scales), xs)
