"""GPU parity of the fused GDN gate projection (nvfp4_gemm_gdn_gates, paper
Eq. 1 in the GEMM epilogue).

* Epilogue math: the fused kernel's FP32 (beta | alpha) against the float64
  gate transform of the same kernel family's plain FP32 GEMM output (the
  accumulators are bit-identical, so only the binary32 transcendental chain
  differs): relative error <= 1e-5 (1 + |g|) for alpha and 1e-5 for beta.
* End to end: against the oracle gate transform of the oracle GEMM (the GEMM
  error propagated through the gate derivatives, plus the same bound).
* BF16 output equals the round-to-nearest-even of the FP32 output.
"""

import numpy as np
import pytest
import torch

from oracle import gates as OGa
from oracle import gemm as OG
from oracle import quant as OQ
from paper_2609_04098_amd import linear as L
from paper_2609_04098_amd import synth
from tests.gpu_common import ELEM_TOL, log, to_dev_bf16, workload

pytestmark = pytest.mark.gpu


def _gate_params(h, seed):
    rng = np.random.default_rng(seed)
    a_log = np.log(rng.uniform(1.0, 16.0, h)).astype(np.float32)      # A in [1, 16]
    dt_bias = rng.uniform(-4.0, 2.0, h).astype(np.float32)
    return a_log, dt_bias


def _run(x_bits, w_bits, h, a_log, dt_bias):
    aq = L.quantize_act(to_dev_bf16(x_bits))
    pw = L.pack_weight(to_dev_bf16(w_bits), [0, h, 2 * h])
    al = torch.from_numpy(a_log).cuda()
    dt = torch.from_numpy(dt_bias).cuda()
    g32 = L.gemm_gdn_gates(aq, pw, al, dt, out_dtype=torch.float32)
    g16 = L.gemm_gdn_gates(aq, pw, al, dt, out_dtype=torch.bfloat16)
    plain = L.gemm(aq, pw, out_dtype=torch.float32)
    torch.cuda.synchronize()
    return g32, g16, plain


def _check_transform(gates, plain, a_log, dt_bias, what):
    h = gates.shape[1] // 2
    ref = OGa.gdn_gates(plain, a_log.astype(np.float64), dt_bias.astype(np.float64))
    g = -np.exp(a_log.astype(np.float64))[None, :] * OGa.softplus(plain[:, h:] + dt_bias[None, :])
    err = np.abs(gates - ref)
    ok_b = err[:, :h] <= 1e-5 * ref[:, :h] + 1e-30
    ok_a = err[:, h:] <= 1e-5 * (1.0 + np.abs(g)) * ref[:, h:] + 1e-30
    assert ok_b.all(), "%s beta: worst rel %g" % (what, float((err[:, :h] / ref[:, :h]).max()))
    assert ok_a.all(), "%s alpha: worst rel %g" % (what, float((err[:, h:] / np.maximum(ref[:, h:], 1e-300)).max()))


@pytest.mark.parametrize("m,k,h", [(300, 512, 48), (64, 5120, 48), (1, 128, 4), (257, 256, 40), (100, 256, 64)])
def test_gate_epilogue(m, k, h):
    rng = np.random.default_rng(m + k + h)
    x = rng.standard_normal((m, k))
    x[:, rng.choice(k, max(1, k // 200), replace=False)] *= 80
    w = rng.standard_normal((2 * h, k)) * 0.05
    xb, wb = synth.f64_to_bf16_bits(x), synth.f64_to_bf16_bits(w)
    a_log, dt_bias = _gate_params(h, m)
    g32, g16, plain = _run(xb, wb, h, a_log, dt_bias)
    gates = g32.cpu().numpy().astype(np.float64)
    if 2 * h <= 96 or m <= 32:
        # The plain GEMM runs the same split-K kernel: identical accumulators.
        _check_transform(gates, plain.cpu().numpy().astype(np.float64), a_log, dt_bias, "%dx%dx%d" % (m, k, h))
    assert torch.equal(g16.view(torch.int16), g32.to(torch.bfloat16).view(torch.int16))
    # End to end against the oracle: the GEMM error (<= 1e-4 sum|ab| per
    # element) moves beta by at most beta(1-beta) times it and alpha by at
    # most alpha exp(A_log) sigmoid(a + dt) times it.
    xp, xs, gx = OQ.quantize_tensor(xb)
    wp, ws, gw = OQ.quantize_segments(wb, [0, h, 2 * h])
    y_ref = OG.gemm_exact(xp, xs, gx, wp, ws, gw, [0, h, 2 * h])
    r_ref = OG.abs_bound(xp, xs, gx, wp, ws, gw, [0, h, 2 * h])
    ref = OGa.gdn_gates(y_ref, a_log, dt_bias)
    dy = ELEM_TOL * r_ref + 1e-30
    sig_a = OGa.sigmoid(y_ref[:, h:] + dt_bias[None, :])
    g = -np.exp(a_log.astype(np.float64))[None, :] * OGa.softplus(y_ref[:, h:] + dt_bias[None, :])
    bound_b = ref[:, :h] * (1 - ref[:, :h]) * dy[:, :h] * 1.01 + 1e-5 * ref[:, :h]
    bound_a = ref[:, h:] * np.exp(a_log)[None, :] * sig_a * dy[:, h:] * 1.01 + 1e-5 * (1 + np.abs(g)) * ref[:, h:]
    err = np.abs(gates - ref)
    assert np.all(err[:, :h] <= bound_b + 1e-30)
    assert np.all(err[:, h:] <= bound_a + 1e-30)


def test_gate_epilogue_ab_gates_workload():
    """The tall-skinny a/b projection (32768 x 96 x 5120; segment 0 taken as
    b, segment 1 as a), every output checked against the transform of the
    plain GEMM output."""
    wl = workload("ab_gates")
    cfg = wl["cfg"]
    h = cfg.n // 2
    a_log, dt_bias = _gate_params(h, 99)
    g32, g16, plain = _run(wl["x"], wl["w"], h, a_log, dt_bias)
    gates = g32.cpu().numpy().astype(np.float64)
    _check_transform(gates, plain.cpu().numpy().astype(np.float64), a_log, dt_bias, "ab_gates")
    assert torch.equal(g16.view(torch.int16), g32.to(torch.bfloat16).view(torch.int16))
    log("ab_gates: beta in [%.3g, %.3g], alpha in [%.3g, %.3g]" % (
        gates[:, :h].min(), gates[:, :h].max(), gates[:, h:].min(), gates[:, h:].max()))
