"""GPU parity of the allocation-free quantizer (nvfp4_quantize_act_noalloc)
against nvfp4_quantize_act with a caller workspace: the same codes, scales
and global scale, bit for bit, on consecutive calls that share the
library's per-device scratch (the second call smaller than the first), in
both scale modes, and against the CPU oracle."""

import numpy as np
import pytest
import torch

from oracle import quant as OQ
from paper_2609_04098_amd import linear as L
from paper_2609_04098_amd import nvfp4 as C
from paper_2609_04098_amd import synth
from tests.gpu_common import log, np_u8, to_dev_bf16

pytestmark = pytest.mark.gpu


def _bits(v):
    return synth.f64_to_bf16_bits(np.asarray(v, dtype=np.float64))


def _x(seed, m, k, ldx=None):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((m, k))
    x[:, rng.choice(k, max(1, k // 200), replace=False)] *= rng.uniform(50, 200)
    bits = _bits(x)
    if ldx is None:
        return bits, to_dev_bf16(bits)
    buf = np.zeros((m, ldx), dtype=np.uint16)
    buf[:, :k] = bits
    return bits, to_dev_bf16(buf)[:, :k]


def _both(x, mode, g_static=None):
    """(noalloc result, workspace result) as (codes, scales, g) device tensors."""
    m, k = x.shape
    out = []
    for noalloc in (True, False):
        codes = torch.full((m, k // 2), 0x5A, dtype=torch.uint8, device="cuda")
        scales = torch.full((m, k // 16), 0xA5, dtype=torch.uint8, device="cuda")
        g = torch.full((1,), -1.0, dtype=torch.float32, device="cuda")
        if g_static is not None:
            g.fill_(float(g_static))
        if noalloc:
            C.nvfp4_quantize_act_noalloc(x, codes, scales, g, mode)
        else:
            ws = torch.empty(C.nvfp4_quantize_act_workspace(m, k), dtype=torch.uint8, device="cuda")
            C.nvfp4_quantize_act(x, codes, scales, g, mode, ws)
        torch.cuda.synchronize()
        out.append((codes, scales, g))
    return out


def _same(a, b, what):
    assert torch.equal(a[0], b[0]), "%s: codes differ" % what
    assert torch.equal(a[1], b[1]), "%s: scales differ" % what
    assert torch.equal(a[2], b[2]), "%s: global scale differs" % what


def test_noalloc_matches_workspace_entry_point_on_consecutive_calls():
    cases = [
        ("mlp_gate_up activation 8192x5120", None),
        ("ragged strided 300x1040 (ldx 1104)", (301, 300, 1040, 1104)),
        ("decode 1x5120 (one-launch path)", (302, 1, 5120, None)),
        ("odd 777x96", (303, 777, 96, None)),
    ]
    for what, spec in cases:
        if spec is None:
            bits = synth.make_x(synth.CONFIGS["mlp_gate_up"])
            x = to_dev_bf16(bits)
        else:
            bits, x = _x(*spec)
        log("noalloc: %s, dynamic" % what)
        a, b = _both(x, C.NVFP4_DYNAMIC)
        _same(a, b, what + " dynamic")
        if spec is not None:
            xp, xs, gx = OQ.quantize_tensor(bits)
            assert np.array_equal(np_u8(a[0]), xp) and np.array_equal(np_u8(a[1]), xs)
            assert np.float32(a[2].item()) == gx
        log("noalloc: %s, static" % what)
        g_static = np.float32(b[2].item() * 0.75)
        a, b = _both(x, C.NVFP4_STATIC, g_static)
        _same(a, b, what + " static")


def test_noalloc_empty_tensor_writes_zero_scale():
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    codes = torch.empty((0, 32), dtype=torch.uint8, device="cuda")
    scales = torch.empty((0, 4), dtype=torch.uint8, device="cuda")
    g = torch.full((1,), 7.0, dtype=torch.float32, device="cuda")
    C.nvfp4_quantize_act_noalloc(x, codes, scales, g, C.NVFP4_DYNAMIC)
    torch.cuda.synchronize()
    assert g.item() == 0.0
