"""Shared helpers of the GPU parity tests: seeded inputs, device upload,
oracle results per workload (cached per session), and the GEMM tolerance.

GEMM tolerance (stated for the FP32 output): per element
|Y - Y_ref| <= 1e-4 * sum_k |a_k w_k| (plus 1e-30 absolute), and relative
Frobenius error <= 1e-5.  BF16 output must equal the round-to-nearest-even of
the same kernel's FP32 output.
"""

import functools
import sys
import time

import numpy as np
import torch

from oracle import gemm as OG
from oracle import quant as OQ
from paper_2609_04098_amd import synth

ELEM_TOL = 1e-4
FROB_TOL = 1e-5


def log(msg):
    sys.stdout.write("[%s] %s\n" % (time.strftime("%H:%M:%S"), msg))
    sys.stdout.flush()


def to_dev_bf16(bits):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to("cuda")


def np_u8(t):
    return t.detach().cpu().numpy().astype(np.uint8)


@functools.lru_cache(maxsize=2)
def workload(name):
    """Inputs and oracle quantization of one named workload (full size)."""
    cfg = synth.CONFIGS[name]
    t0 = time.time()
    x = synth.make_x(cfg)
    w = synth.make_w(cfg)
    log("%s: inputs drawn in %.1fs" % (name, time.time() - t0))
    t0 = time.time()
    xp, xs, gx = OQ.quantize_tensor(x)
    wp, ws, gw = OQ.quantize_segments(w, cfg.seg_offsets)
    log("%s: oracle quantization in %.1fs" % (name, time.time() - t0))
    return dict(cfg=cfg, x=x, w=w, xp=xp, xs=xs, gx=gx, wp=wp, ws=ws, gw=gw)


def check_gemm(y32, y_ref, r_ref, what=""):
    """Assert the stated GEMM tolerance (float64 numpy arrays)."""
    err = np.abs(y32 - y_ref)
    bad = err > ELEM_TOL * r_ref + 1e-30
    assert not bad.any(), "%s: %d elements over 1e-4*sum|ab|; worst ratio %g" % (
        what, int(bad.sum()), float((err / np.maximum(r_ref, 1e-300)).max()))
    den = np.linalg.norm(y_ref)
    rel = np.linalg.norm(y32 - y_ref) / den if den > 0 else np.linalg.norm(y32)
    assert rel <= FROB_TOL, "%s: relative Frobenius error %g" % (what, rel)
    return rel


def bf16_rne_of(y32_dev):
    """RNE bf16 of an fp32 device tensor, as uint16 bits (test-side check)."""
    return y32_dev.to(torch.bfloat16).view(torch.int16).cpu().numpy().view(np.uint16)
