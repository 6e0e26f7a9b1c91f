"""GPU parity of the fused act-quant + narrow GEMM (nvfp4_quantize_gemm).

The fused call must equal nvfp4_quantize_act followed by nvfp4_gemm: the
activation codes, scales and G_A bit for bit (and equal to the CPU oracle),
and Y bit for bit where both paths sum in the same order (N <= 96 and
K % 64 == 0: the split-K GEMM), else within the GEMM tolerance of the
oracle (tests/gpu_common.py)."""

import numpy as np
import pytest
import torch

from oracle import gemm as OG
from oracle import quant as OQ
from paper_2609_04098_amd import linear as L
from paper_2609_04098_amd import synth
from tests.gpu_common import check_gemm, log, np_u8, to_dev_bf16, workload

pytestmark = pytest.mark.gpu


def bits_of(v):
    return synth.f64_to_bf16_bits(np.asarray(v, dtype=np.float64))


def _xw(rng, m, n, k):
    x = rng.standard_normal((m, k))
    x[:, rng.choice(k, max(1, k // 200), replace=False)] *= 100.0
    w = rng.standard_normal((n, k)) * 0.05
    return bits_of(x), bits_of(w)


def run_both(x_bits, w_bits, offs, g=None, ldx=None):
    m, k = x_bits.shape
    n = w_bits.shape[0]
    if ldx is None:
        x = to_dev_bf16(x_bits)
    else:
        buf = np.zeros((m, ldx), dtype=np.uint16)
        buf[:, :k] = x_bits
        x = to_dev_bf16(buf)[:, :k]
    pw = L.pack_weight(to_dev_bf16(w_bits), offs)
    aq_ref = L.quantize_act(x, g=g)
    y_ref = L.gemm(aq_ref, pw, out_dtype=torch.float32)
    aq = L.alloc_act(m, k, x.device)
    y32, g32 = L.quantize_gemm(x, pw, g=g, out_dtype=torch.float32, act_out=aq)
    y16, _ = L.quantize_gemm(x, pw, g=g, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    return aq_ref, y_ref, aq, y32, g32, y16


def check_case(x_bits, w_bits, offs, g=None, ldx=None, same_order=True):
    aq_ref, y_ref, aq, y32, g32, y16 = run_both(x_bits, w_bits, offs, g, ldx)
    ref_p, ref_s, ref_g = OQ.quantize_tensor(x_bits, g=None if g is None else np.float32(g))
    assert np.float32(g32.item()) == ref_g == np.float32(aq.g.item())
    np.testing.assert_array_equal(np_u8(aq.codes), ref_p)
    np.testing.assert_array_equal(np_u8(aq.scales), ref_s)
    if same_order:
        assert torch.equal(y32, y_ref), "fused and unfused GEMM sums differ"
    wp, ws, gw = OQ.quantize_segments(w_bits, offs)
    y_or = OG.gemm_exact(ref_p, ref_s, ref_g, wp, ws, gw, offs)
    r_or = OG.abs_bound(ref_p, ref_s, ref_g, wp, ws, gw, offs)
    check_gemm(y32.cpu().numpy().astype(np.float64), y_or, r_or, "fused %s" % (x_bits.shape,))
    assert torch.equal(y16.view(torch.int16), y32.to(torch.bfloat16).view(torch.int16))


@pytest.mark.parametrize("m,n,k,offs", [
    (257, 96, 512, [0, 48, 96]),          # 48 + 48 segments in one tile, ragged M
    (100, 72, 320, [0, 40, 72]),          # N not a multiple of 32, 5 chunks over 4 waves
    (33, 90, 128, [0, 30, 90]),           # fewer chunks than waves
    (1, 33, 64, [0, 33]),                 # one row, one chunk
    (300, 96, 5184, [0, 48, 96]),         # 81 chunks over 4 waves
])
def test_quantize_gemm_matches_unfused(m, n, k, offs):
    rng = np.random.default_rng(m * 5 + n * 3 + k)
    x, w = _xw(rng, m, n, k)
    check_case(x, w, offs)                                  # dynamic G
    check_case(x, w, offs, g=np.float32(2688.0 / 50.0))    # static G, saturating outliers


def test_quantize_gemm_wide_tile_strided_rows():
    rng = np.random.default_rng(7)
    x, w = _xw(rng, 150, 128, 256)
    # N in (96, 128]: the unfused path is the LDS GEMM (another summation order)
    check_case(x, w, [0, 100, 128], ldx=272, same_order=False)


def test_quantize_gemm_edge_values():
    rng = np.random.default_rng(11)
    x = rng.standard_normal((64, 128))
    x[0] = 0.0                            # zero row
    x[1, :16] = 0.0                       # zero block
    x[2, :16] *= 1e-4
    x[2, 16] = 3e3                        # subnormal-scale block beside an outlier
    xb = bits_of(x)
    xb[3, ::3] = 0x8000                   # signed zeros
    w = bits_of(rng.standard_normal((96, 128)) * 0.05)
    check_case(xb, w, [0, 48, 96])
    check_case(xb, w, [0, 48, 96], g=np.float32(3e30))
    check_case(np.zeros((40, 128), dtype=np.uint16), w, [0, 48, 96])   # all-zero X: G = 0, Y = 0


def test_quantize_gemm_full_ab_gates():
    wl = workload("ab_gates")
    cfg = wl["cfg"]
    log("ab_gates: fused quantize + GEMM on GPU")
    aq_ref, y_ref, aq, y32, g32, y16 = run_both(wl["x"], wl["w"], cfg.seg_offsets)
    assert np.float32(g32.item()) == wl["gx"]
    np.testing.assert_array_equal(np_u8(aq.scales), wl["xs"])
    np.testing.assert_array_equal(np_u8(aq.codes), wl["xp"])
    assert torch.equal(y32, y_ref)
    assert torch.equal(y16.view(torch.int16), y32.to(torch.bfloat16).view(torch.int16))
    rng = np.random.default_rng(5)
    rows = np.array(sorted(set(list(range(8)) + list(range(cfg.m - 8, cfg.m)) +
                               list(rng.choice(np.arange(8, cfg.m - 8), 16, replace=False)))))
    args = (wl["xp"], wl["xs"], wl["gx"], wl["wp"], wl["ws"], wl["gw"], cfg.seg_offsets)
    check_gemm(y32[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64),
               OG.gemm_f64(*args, rows=rows), OG.abs_bound(*args, rows=rows), "ab_gates fused")


# ---------------------------------------------------------------- decode path
# M <= 32 with N > 128: one launch in which every workgroup quantizes X into
# its LDS and runs the M <= 32 split-K GEMM on it (activations up to 24 KB
# quantized), else the quantizer and the same GEMM; Y must equal the unfused
# quantize + GEMM bit for bit either way.

@pytest.mark.parametrize("m,n,k,offs", [
    (1, 300, 1024, [0, 300]),              # one row, ragged N
    (7, 520, 5120, [0, 260, 520]),         # hidden width, two segments
    (32, 200, 128, [0, 72, 200]),          # 2 chunks < 4 waves
    (17, 4100, 256, [0, 4000, 4100]),      # many workgroups, few blocks each
    (5, 129, 64, [0, 129]),                # one chunk, N just past the narrow limit
    (20, 300, 2560, [0, 150, 300]),        # 28.8 KB quantized: the two-launch decode path
    (3, 640, 5120, [0, 320, 640]),         # M * K = 15360: the largest one-launch case at the hidden width
    (4, 640, 5120, [0, 320, 640]),         # M * K = 20480: the smallest two-launch case there
    (8, 700, 2048, [0, 350, 700]),         # the most rows with per-wave activation rings
    (9, 700, 2048, [0, 350, 700]),         # the fewest rows with the shared activation ring
])
def test_quantize_gemm_decode_matches_unfused(m, n, k, offs):
    rng = np.random.default_rng(m * 11 + n * 7 + k)
    x, w = _xw(rng, m, n, k)
    check_case(x, w, offs)                                  # dynamic G
    check_case(x, w, offs, g=np.float32(2688.0 / 40.0))    # static G, saturating outliers
    check_case(x, w, offs, ldx=k + 64)                      # strided rows


def test_quantize_gemm_decode_edge_values():
    rng = np.random.default_rng(12)
    x = rng.standard_normal((9, 256))
    x[0] = 0.0
    x[1, :16] = 0.0
    x[2, :16] *= 1e-4
    x[2, 16] = 3e3
    xb = bits_of(x)
    xb[3, ::3] = 0x8000
    w = bits_of(rng.standard_normal((160, 256)) * 0.05)
    check_case(xb, w, [0, 100, 160])
    check_case(xb, w, [0, 100, 160], g=np.float32(3e30))
    check_case(np.zeros((4, 256), dtype=np.uint16), w, [0, 100, 160])


@pytest.mark.parametrize("m", [1, 7, 32])
def test_quantize_gemm_decode_full_gate_up(m):
    """Decode rows against the full gate/up weight (34816 x 5120, two
    segments): codes, scales and G equal the oracle's, Y equals the unfused
    path bit for bit and the oracle within the GEMM tolerance on every
    element; three calls on one workspace agree."""
    wl = workload("decode_m32")
    cfg = wl["cfg"]
    x_bits = wl["x"][:m]
    x = to_dev_bf16(x_bits)
    pw = L.pack_weight(to_dev_bf16(wl["w"]), cfg.seg_offsets)
    log("decode m=%d: fused quantize + GEMM on GPU" % m)
    aq_ref = L.quantize_act(x)
    y_ref = L.gemm(aq_ref, pw, out_dtype=torch.float32)
    ws = L.quantize_gemm_workspace(m, cfg.n, cfg.k, x.device)
    aq = L.alloc_act(m, cfg.k, x.device)
    ys = []
    for i in range(3):
        y32, g32 = L.quantize_gemm(x, pw, out_dtype=torch.float32, act_out=aq if i == 0 else None, workspace=ws)
        ys.append(y32)
    y16, _ = L.quantize_gemm(x, pw, out_dtype=torch.bfloat16, workspace=ws)
    torch.cuda.synchronize()
    xp, xs, gx = OQ.quantize_tensor(x_bits)
    assert np.float32(g32.item()) == gx == np.float32(aq.g.item())
    np.testing.assert_array_equal(np_u8(aq.codes), xp)
    np.testing.assert_array_equal(np_u8(aq.scales), xs)
    for y32 in ys:
        assert torch.equal(y32, y_ref), "fused decode GEMM differs from the unfused path"
    assert torch.equal(y16.view(torch.int16), ys[0].to(torch.bfloat16).view(torch.int16))
    args = (xp, xs, gx, wl["wp"], wl["ws"], wl["gw"], cfg.seg_offsets)
    rel = check_gemm(ys[0].cpu().numpy().astype(np.float64), OG.gemm_f64(*args), OG.abs_bound(*args),
                     "decode m=%d" % m)
    log("decode m=%d: relative Frobenius error %.3g" % (m, rel))
