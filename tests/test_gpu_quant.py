"""GPU parity of the activation quantizer (nvfp4_quantize_act) and the weight
prepack (nvfp4_pack_weight / nvfp4_unpack_weight) against the CPU oracle:
codes, block scales and global scales must match bit for bit."""

import json
import os

import numpy as np
import pytest
import torch

from oracle import quant as OQ
from paper_2609_04098_amd import linear as L
from paper_2609_04098_amd import nvfp4 as C
from paper_2609_04098_amd import synth
from tests.gpu_common import log, np_u8, to_dev_bf16, workload

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def bits_of(v):
    return synth.f64_to_bf16_bits(np.asarray(v, dtype=np.float64))


def gpu_act(x_bits, g=None, ldx=None):
    m, k = x_bits.shape
    if ldx is None:
        x = to_dev_bf16(x_bits)
    else:                                   # strided rows: a view into a wider buffer
        buf = np.zeros((m, ldx), dtype=np.uint16)
        buf[:, :k] = x_bits
        x = to_dev_bf16(buf)[:, :k]
    aq = L.quantize_act(x, g=g)
    torch.cuda.synchronize()
    return np_u8(aq.codes), np_u8(aq.scales), np.float32(aq.g.cpu().item())


def assert_act_matches(x_bits, g=None, ldx=None):
    codes, scales, g_dev = gpu_act(x_bits, g, ldx)
    ref_p, ref_s, ref_g = OQ.quantize_tensor(x_bits, g=None if g is None else np.float32(g))
    assert g_dev == ref_g, (g_dev, ref_g)
    np.testing.assert_array_equal(scales, ref_s)
    np.testing.assert_array_equal(codes, ref_p)


# ----------------------------------------------------------------- activation

def test_act_quant_tiny_workload():
    x = synth.make_x(synth.CONFIGS["tiny"])
    assert_act_matches(x)


def test_act_quant_hand_worked_example():
    with open(os.path.join(HERE, "golden", "worked_block.json")) as f:
        ex = json.load(f)
    codes, scales, _ = gpu_act(bits_of([ex["x"]]), g=ex["g"])
    assert scales[0].tolist() == ex["scale_codes"]
    assert OQ.unpack_nibbles(codes)[0].tolist() == ex["codes"]


def test_act_quant_edge_cases():
    rng = np.random.default_rng(100)
    x = rng.standard_normal((40, 96))
    x[0] = 0.0                              # all-zero row
    x[1, :16] = 0.0                         # all-zero block
    x[2, :16] *= 1e-4                       # subnormal-scale block next to an outlier
    x[2, 16] = 3e3
    x[3, ::3] = -0.0                        # signed zeros
    x[4, :] = -1e-35                        # tiny negatives
    xb = bits_of(x)
    xb[3, ::3] = 0x8000
    xb[5, :16] = np.arange(1, 17, dtype=np.uint16) * 7        # bf16 subnormals (block max among them)
    xb[5, 16:32] = 0x8000 | (np.arange(1, 17, dtype=np.uint16) * 5)   # negative subnormals
    assert_act_matches(xb)
    assert_act_matches(xb, ldx=128)         # strided rows
    # static scale from a smaller calibration amax: scales and codes saturate
    assert_act_matches(xb, g=np.float32(2688.0 / 50.0))
    assert_act_matches(xb, g=np.float32(1.0))
    assert_act_matches(xb, g=np.float32(3e30))
    assert_act_matches(xb, g=np.float32(3.0e38))   # subnormal blocks get non-zero scales
    assert_act_matches(xb, g=np.float32(1e20))     # most values far beyond the range: saturation


def test_act_quant_small_and_two_pass_paths_agree_on_edge_cases():
    """Activations of at most 4096 blocks take the one-launch quantizer; the
    same edge rows repeated past that size take the two-pass one."""
    rng = np.random.default_rng(101)
    x = rng.standard_normal((40, 96))
    x[0] = 0.0
    x[2, :16] *= 1e-4
    x[2, 16] = 3e3
    x[4, :] = -1e-35
    xb = bits_of(x)
    xb[3, ::3] = 0x8000
    big = np.tile(xb, (20, 1))                    # 800 x 96: 4800 blocks
    for t in (xb, big):
        assert_act_matches(t)
        assert_act_matches(t, ldx=128)
        assert_act_matches(t, g=np.float32(2688.0 / 50.0))
        assert_act_matches(t, g=np.float32(3e30))
    z = np.zeros((4200, 16), dtype=np.uint16)     # denormal amax, two-pass path
    z[1, 3] = 0x0001
    assert_act_matches(z)


@pytest.mark.parametrize("m,k", [(256, 256), (4097, 16), (1, 65536), (1, 65552), (64, 1040)])
def test_act_quant_one_launch_boundary(m, k):
    # 4096 blocks (256 x 256, one row of 65536) is the largest activation
    # the one-launch quantizer takes; 4097 blocks go to the two passes;
    # 64 x 1040 (4160 blocks) is a two-pass shape whose K is not a multiple
    # of 32.
    rng = np.random.default_rng(m + k)
    x = rng.standard_normal((m, k))
    x[:, rng.choice(k, max(1, k // 200), replace=False)] *= 100.0
    xb = bits_of(x)
    assert_act_matches(xb)
    assert_act_matches(xb, g=np.float32(2688.0 / 50.0))


def test_act_quant_special_tensors():
    assert_act_matches(np.zeros((8, 32), dtype=np.uint16))            # G = 0
    z = np.zeros((4, 16), dtype=np.uint16)
    z[1, 3] = 0x0001                                                  # denormal amax: G saturates
    z[2, 5] = 0x8003
    assert_act_matches(z)
    assert_act_matches(bits_of(np.random.default_rng(1).standard_normal((1, 16))))


def test_act_quant_every_bf16_magnitude():
    # every positive bf16 value below 3 next to a block max of 3, under G = 1
    # (block scale 0.5), and the same tensor in dynamic mode
    amax = bits_of([3.0])[0]
    below = np.arange(0x0001, int(amax), dtype=np.uint16)
    pad = (-len(below)) % 15
    below = np.concatenate([below, np.zeros(pad, dtype=np.uint16)]).reshape(-1, 15)
    xb = np.concatenate([np.full((below.shape[0], 1), amax, dtype=np.uint16), below], axis=1)
    xb = xb[: (xb.shape[0] // 4) * 4].reshape(-1, 64)
    xb[::2] |= 0x8000
    assert_act_matches(xb, g=np.float32(1.0))
    assert_act_matches(xb)


def test_act_quant_exact_ties():
    # block maxima at 6 x (E4M3 midpoints) and elements at (E2M1 midpoints) x S
    from oracle.formats import E4M3_GRID
    mids = (E4M3_GRID[:-1] + E4M3_GRID[1:]) / 2
    rows = []
    for m in mids:
        blk = np.zeros(16)
        blk[0] = 6.0 * m
        s = E4M3_GRID[np.searchsorted(E4M3_GRID, m)]          # one of the neighbours
        blk[1:8] = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]) * s
        blk[8:15] = -blk[1:8]
        rows.append(blk)
    xb = bits_of(np.array(rows))
    assert_act_matches(xb, g=np.float32(1.0))
    assert_act_matches(xb, g=np.float32(0.5))


def near_midpoint_blocks(g, rng_scales):
    """Blocks [amax, x, -x, 0, ...] whose scale is S and whose x has |x| G / S
    within 2^-19 (relative) of an E2M1 rounding midpoint without being on it."""
    from oracle.formats import E4M3_GRID, bf16_bits_to_f64
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    s = E4M3_GRID[rng_scales]
    target = mids[None, :] * s[:, None] / float(g)
    base = bits_of(target).astype(np.int64)
    blocks = []
    for d in (-1, 0, 1):
        xb = (base + d).astype(np.uint16)
        q = bf16_bits_to_f64(xb) * float(g) / s[:, None]          # exact: 8 x 24 bits, S a power-of-two multiple
        rel = np.abs(q - mids[None, :]) / mids[None, :]
        for i, j in zip(*np.nonzero((rel > 0) & (rel < 2.0 ** -19))):
            blk = np.zeros(16, dtype=np.uint16)
            blk[0] = bits_of([6.0 * s[i] / float(g)])[0]           # rounds back to S
            blk[1] = xb[i, j]
            blk[2] = xb[i, j] | 0x8000
            blocks.append(blk)
    return blocks


def test_act_quant_near_midpoints():
    """Elements whose exact |x| G / S lies within 2^-19 of an E2M1 midpoint,
    on either side of it: a quotient rounded anywhere before the decision
    could land on the wrong side."""
    rng = np.random.default_rng(2024)
    found = 0
    for trial in range(400):
        g = np.float32(rng.uniform(1.0, 2.0) * 2.0 ** int(rng.integers(-4, 5)))
        blocks = near_midpoint_blocks(g, np.arange(40, 120))
        if not blocks:
            continue
        found += len(blocks)
        xb = np.concatenate(blocks).reshape(-1, 16 * len(blocks))
        assert_act_matches(xb, g=g)
    assert found >= 20, found


def test_act_quant_empty():
    g = torch.full((1,), 7.0, dtype=torch.float32, device="cuda")
    ws = L.act_workspace(0, 64, "cuda")
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    codes = torch.empty((0, 32), dtype=torch.uint8, device="cuda")
    scales = torch.empty((0, 4), dtype=torch.uint8, device="cuda")
    C.nvfp4_quantize_act(x, codes, scales, g, C.NVFP4_DYNAMIC, ws)
    torch.cuda.synchronize()
    assert g.item() == 0.0


def test_act_quant_does_not_write_past_outputs():
    x = bits_of(np.random.default_rng(2).standard_normal((33, 48)))
    xd = to_dev_bf16(x)
    codes = torch.full((33 * 24 + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    scales = torch.full((33 * 3 + 64,), 0x5A, dtype=torch.uint8, device="cuda")
    g = torch.zeros(1, dtype=torch.float32, device="cuda")
    ws = L.act_workspace(33, 48, "cuda")
    C.nvfp4_quantize_act(xd, codes, scales, g, C.NVFP4_DYNAMIC, ws)
    torch.cuda.synchronize()
    assert np.all(np_u8(codes[33 * 24:]) == 0xA5) and np.all(np_u8(scales[33 * 3:]) == 0x5A)


@pytest.mark.parametrize("name", synth.CONFIG_ORDER)
def test_act_quant_full_workloads(name):
    wl = workload(name)
    log("%s: act quant on GPU" % name)
    codes, scales, g = gpu_act(wl["x"])
    assert g == wl["gx"]
    np.testing.assert_array_equal(scales, wl["xs"])
    np.testing.assert_array_equal(codes, wl["xp"])


# --------------------------------------------------------------------- weight

def gpu_pack(w_bits, offs, g_seg=None):
    w = to_dev_bf16(w_bits)
    pw = L.pack_weight(w, offs, g_seg)
    codes, scales = L.unpack_weight(pw)
    torch.cuda.synchronize()
    return np_u8(codes), np_u8(scales), pw.g_seg.cpu().numpy()


def assert_pack_matches(w_bits, offs, g_seg=None):
    codes, scales, gs = gpu_pack(w_bits, offs, g_seg)
    rp, rs, rg = OQ.quantize_segments(w_bits, offs, g_seg)
    np.testing.assert_array_equal(gs, np.array(rg, dtype=np.float32))
    np.testing.assert_array_equal(scales, rs)
    np.testing.assert_array_equal(codes, rp)


def test_pack_weight_ragged_shapes():
    rng = np.random.default_rng(200)
    for n, k, offs in [(100, 80, [0, 37, 100]), (96, 5120 // 4, [0, 48, 96]), (33, 272, [0, 1, 2, 33]),
                       (8, 16, [0, 8]), (300, 512, [0, 100, 150, 151, 300])]:
        w = rng.standard_normal((n, k)) * 0.02
        w[:, 0] *= 40
        assert_pack_matches(bits_of(w), offs)
        assert_pack_matches(bits_of(w), offs, [np.float32(1000.0 + i) for i in range(len(offs) - 1)])


def test_pack_weight_segments_of_very_different_scale():
    rng = np.random.default_rng(201)
    w = np.concatenate([rng.standard_normal((32, 64)) * 1e-3, rng.standard_normal((32, 64)) * 50.0,
                        np.zeros((32, 64))])
    assert_pack_matches(bits_of(w), [0, 32, 64, 96])


@pytest.mark.parametrize("name", synth.CONFIG_ORDER)
def test_pack_weight_full_workloads(name):
    wl = workload(name)
    log("%s: weight pack on GPU" % name)
    codes, scales, gs = gpu_pack(wl["w"], wl["cfg"].seg_offsets)
    np.testing.assert_array_equal(gs, np.array(wl["gw"], dtype=np.float32))
    np.testing.assert_array_equal(scales, wl["ws"])
    np.testing.assert_array_equal(codes, wl["wp"])
