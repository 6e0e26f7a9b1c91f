"""GPU parity of the NVFP4 GEMM (nvfp4_gemm_with_workspace, and nvfp4_gemm
where the two differ) against the CPU oracle.

FP32 output: per element |Y - Y_ref| <= 1e-4 * sum_k |a_k w_k| and relative
Frobenius error <= 1e-5 (tests/gpu_common.py).  BF16 output: equal to the
round-to-nearest-even of the same kernel's FP32 output.  Small and ragged
shapes are checked on every element; the full workloads on sampled rows
(all columns of each sampled row)."""

import numpy as np
import pytest
import torch

from oracle import gemm as OG
from oracle import quant as OQ
from paper_2609_04098_amd import linear as L
from paper_2609_04098_amd import nvfp4 as C
from paper_2609_04098_amd import synth
from tests.gpu_common import bf16_rne_of, check_gemm, log, np_u8, to_dev_bf16, workload

pytestmark = pytest.mark.gpu


def bits_of(v):
    return synth.f64_to_bf16_bits(np.asarray(v, dtype=np.float64))


def run_gpu(x_bits, w_bits, offs, ldy=None, use_ws=True):
    """Quantize, pack and multiply on the GPU; returns (y32, y16 bits, aq, pw).
    use_ws=False: through nvfp4_gemm (no workspace)."""
    m, n = x_bits.shape[0], w_bits.shape[0]
    aq = L.quantize_act(to_dev_bf16(x_bits))
    pw = L.pack_weight(to_dev_bf16(w_bits), offs)
    ldy = n if ldy is None else ldy
    y32 = torch.empty((m, ldy), dtype=torch.float32, device="cuda")[:, :n]
    y16 = torch.empty((m, ldy), dtype=torch.bfloat16, device="cuda")[:, :n]
    mul = L.gemm if use_ws else L.gemm_no_workspace
    mul(aq, pw, out=y32)
    mul(aq, pw, out=y16)
    torch.cuda.synchronize()
    return y32, y16, aq, pw


def oracle_all(x_bits, w_bits, offs):
    xp, xs, gx = OQ.quantize_tensor(x_bits)
    wp, ws, gw = OQ.quantize_segments(w_bits, offs)
    y = OG.gemm_exact(xp, xs, gx, wp, ws, gw, offs)
    r = OG.abs_bound(xp, xs, gx, wp, ws, gw, offs)
    return y, r


def check_small(x_bits, w_bits, offs, ldy=None, what=""):
    y32, y16, _, _ = run_gpu(x_bits, w_bits, offs, ldy)
    y_ref, r_ref = oracle_all(x_bits, w_bits, offs)
    check_gemm(y32.cpu().numpy().astype(np.float64), y_ref, r_ref, what)
    np.testing.assert_array_equal(y16.contiguous().view(torch.int16).cpu().numpy().view(np.uint16),
                                  bf16_rne_of(y32.contiguous()))


def _xw(rng, m, n, k, outliers=True):
    x = rng.standard_normal((m, k))
    if outliers:
        x[:, rng.choice(k, max(1, k // 200), replace=False)] *= 100.0
    w = rng.standard_normal((n, k)) * 0.02
    return bits_of(x), bits_of(w)


def test_gemm_tiny_workload():
    cfg = synth.CONFIGS["tiny"]
    check_small(synth.make_x(cfg), synth.make_w(cfg), cfg.seg_offsets, what="tiny")


@pytest.mark.parametrize("m,n,k,offs", [
    (100, 72, 80, [0, 40, 72]),            # K % 64 == 16: unaligned-K path, ragged M/N
    (300, 300, 320, [0, 1, 299, 300]),     # 2 x 2 tiles, K % 256 != 0, 1-column segments
    (257, 96, 512, [0, 48, 96]),           # tall-skinny path, 48 + 48 segments in one tile
    (64, 40, 48, [0, 40]),                 # tall-skinny path, N not a multiple of 32
    (1, 33, 16, [0, 33]),                  # single row, single block
    (300, 96, 5184, [0, 48, 96]),          # tall-skinny split-K: 81 chunks over 4 waves
    (70, 64, 192, [0, 64]),                # tall-skinny split-K: fewer chunks than waves
    (33, 90, 80, [0, 30, 90]),             # tall-skinny split-K, unaligned K, ragged N
    (513, 520, 1024, [0, 100, 200, 300, 400, 500, 510, 515, 520]),   # 8 segments
    (32, 520, 5120, [0, 260, 520]),        # small-M split-K: 80 chunks over 4 waves, ragged N
    (1, 300, 1040, [0, 300]),              # small-M, one row, K % 64 != 0
    (17, 4100, 128, [0, 4000, 4100]),      # small-M, many column tiles, 2 chunks < 4 waves
    (777, 1300, 384, [0, 500, 1300]),      # prefill path: 4 x 6 tiles of 256 x 256, ragged M and N
    (40, 96, 768, [0, 48, 96]),            # tall-skinny split-K: 3 chunks per wave (= ring stages)
    (9, 200, 320, [0, 100, 200]),          # small-M, shared activation ring: 5 chunks, 3 waves idle in step 2
    (8, 200, 320, [0, 100, 200]),          # small-M, private activation rings (the largest such M)
    (5, 200, 1024, [0, 100, 200]),         # small-M split-K: 4 chunks per wave (one refill)
    (9, 64, 960, [0, 64]),                 # split-K: 15 chunks, 4/4/4/3 per wave
    (33, 520, 1024, [0, 260, 520]),        # one row past the small-M split-K limit: 256 x 256 tiles, 33 rows
    (300, 97, 512, [0, 48, 97]),           # one column past the tall-skinny limit: one partial tile column
])
def test_gemm_ragged_shapes(m, n, k, offs):
    rng = np.random.default_rng(m * 7 + n * 3 + k)
    x, w = _xw(rng, m, n, k)
    check_small(x, w, offs, what="%dx%dx%d" % (m, n, k))


@pytest.mark.parametrize("k", [128, 512])
@pytest.mark.parametrize("use_ws", [False, True])
def test_gemm_tail_columns(k, use_ws):
    # 2 x 130 tiles of 256 x 256: on a 256-CU device the 4 tiles past two
    # full rounds (two tile columns) run as a second launch: 256 x 128 tiles
    # (nvfp4_gemm, or K % 512 != 0), or, with a workspace and K = 512, the
    # square tiles as two K halves (FP32 partials, then the summing pass).
    # Ragged M and N (a tail 357 columns wide: the partial-sum rows are
    # padded to 360) inside that tail.  K = 512 runs the scale super-stage
    # kernel for the first launch.  Every element is checked.
    rng = np.random.default_rng(304 + k)
    m, n = 300, 129 * 256 + 101
    x, w = _xw(rng, m, n, k)
    offs = [0, 20000, 33000, n]
    y32, y16, _, _ = run_gpu(x, w, offs, use_ws=use_ws)
    xp, xs, gx = OQ.quantize_tensor(x)
    wp, ws, gw = OQ.quantize_segments(w, offs)
    y_ref = OG.gemm_f64(xp, xs, gx, wp, ws, gw, offs)
    r_ref = OG.abs_bound(xp, xs, gx, wp, ws, gw, offs)
    check_gemm(y32.cpu().numpy().astype(np.float64), y_ref, r_ref, "tail K=%d ws=%s" % (k, use_ws))
    np.testing.assert_array_equal(y16.contiguous().view(torch.int16).cpu().numpy().view(np.uint16),
                                  bf16_rne_of(y32.contiguous()))
    kernels = L.gemm_kernels(m, n, k, with_workspace=use_ws)
    log("tail K=%d ws=%s: launches %s" % (k, use_ws, kernels))
    if torch.cuda.get_device_properties(0).multi_processor_count == 256:
        assert len(kernels) == 2
        assert ("two K halves" in kernels[1]) == (use_ws and k % 512 == 0)


def test_gemm_last_round_as_k_halves_one_tile():
    """One tile row, (CUs + 1) tile columns: the single tile of the last
    round runs as two K halves on two CUs (with a workspace), ragged segment
    boundaries inside it; every element against the oracle, and the bf16
    output equal to RNE of the FP32 output.  The workspace path and
    nvfp4_gemm agree on every column outside that tile bit for bit."""
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    rng = np.random.default_rng(306)
    m, n, k = 256, (ncu + 1) * 256, 1024
    x, w = _xw(rng, m, n, k)
    offs = [0, 1000, n - 100, n]
    need = C.nvfp4_gemm_workspace(m, n, k)
    assert need == 2 * m * 256 * 4
    y32, y16, aq, pw = run_gpu(x, w, offs)
    y_nows = L.gemm_no_workspace(aq, pw, out_dtype=torch.float32)
    torch.cuda.synchronize()
    xp, xs, gx = OQ.quantize_tensor(x)
    wp, ws, gw = OQ.quantize_segments(w, offs)
    y_ref = OG.gemm_f64(xp, xs, gx, wp, ws, gw, offs)
    r_ref = OG.abs_bound(xp, xs, gx, wp, ws, gw, offs)
    check_gemm(y32.cpu().numpy().astype(np.float64), y_ref, r_ref, "K halves, one tile")
    check_gemm(y_nows.cpu().numpy().astype(np.float64), y_ref, r_ref, "no workspace")
    np.testing.assert_array_equal(y16.contiguous().view(torch.int16).cpu().numpy().view(np.uint16),
                                  bf16_rne_of(y32.contiguous()))
    assert torch.equal(y32[:, : n - 256], y_nows[:, : n - 256])
    # strided output rows: the same values
    y_str = torch.empty((m, n + 8), dtype=torch.float32, device="cuda")[:, :n]
    L.gemm(aq, pw, out=y_str)
    torch.cuda.synchronize()
    assert torch.equal(y_str, y32)
    # a workspace one byte short is refused
    with pytest.raises(C.Nvfp4Error):
        L.gemm(aq, pw, out=y32, workspace=torch.empty(need - 1, dtype=torch.uint8, device="cuda"))


def test_gemm_super_stage_every_element():
    # The scale super-stage kernel (K % 256 == 0) over 5 x 6 tiles with
    # ragged M and N, 32 chunks (8 super-stages), every element checked.
    rng = np.random.default_rng(305)
    m, n, k = 1100, 1500, 2048
    x, w = _xw(rng, m, n, k)
    offs = [0, 700, 1500]
    y32, y16, _, _ = run_gpu(x, w, offs)
    xp, xs, gx = OQ.quantize_tensor(x)
    wp, ws, gw = OQ.quantize_segments(w, offs)
    y_ref = OG.gemm_f64(xp, xs, gx, wp, ws, gw, offs)
    r_ref = OG.abs_bound(xp, xs, gx, wp, ws, gw, offs)
    check_gemm(y32.cpu().numpy().astype(np.float64), y_ref, r_ref, "super-stage")
    np.testing.assert_array_equal(y16.contiguous().view(torch.int16).cpu().numpy().view(np.uint16),
                                  bf16_rne_of(y32.contiguous()))
    assert "Super" in L.gemm_kernels(m, n, k)[0]


def test_gemm_strided_output():
    rng = np.random.default_rng(300)
    x, w = _xw(rng, 70, 136, 256)
    check_small(x, w, [0, 64, 136], ldy=256, what="ldy")


@pytest.mark.parametrize("ldy,col0", [(768, 0), (771, 0), (776, 1), (776, 8)])
def test_gemm_bf16_rows_staged_or_not(ldy, col0):
    # The prefill kernel's bf16 epilogue stages whole wave blocks through
    # LDS and stores 16 bytes of a row per lane when every output row starts
    # on a 16-byte boundary (ldy = 768, or 776 at an 8-column offset), and
    # stores element by element otherwise (ldy = 771; or the output shifted
    # by one column).  Segment boundaries on multiples of 256 keep every
    # wave block in one segment.  Every bf16 value must be RNE of the FP32
    # output, and nothing outside the output may be written.
    rng = np.random.default_rng(307)
    m, n, k = 512, 768, 256
    x, w = _xw(rng, m, n, k)
    offs = [0, 256, n]
    aq = L.quantize_act(to_dev_bf16(x))
    pw = L.pack_weight(to_dev_bf16(w), offs)
    y32 = L.gemm(aq, pw, out_dtype=torch.float32)
    big = torch.full((m, ldy), -7.0, dtype=torch.bfloat16, device="cuda")
    y16 = big[:, col0:col0 + n]
    assert y16.stride(0) == ldy
    L.gemm(aq, pw, out=y16)
    torch.cuda.synchronize()
    xp, xs, gx = OQ.quantize_tensor(x)
    wp, ws, gw = OQ.quantize_segments(w, offs)
    check_gemm(y32.cpu().numpy().astype(np.float64), OG.gemm_f64(xp, xs, gx, wp, ws, gw, offs),
               OG.abs_bound(xp, xs, gx, wp, ws, gw, offs), "ldy %d col0 %d" % (ldy, col0))
    np.testing.assert_array_equal(y16.contiguous().view(torch.int16).cpu().numpy().view(np.uint16),
                                  bf16_rne_of(y32))
    rest = torch.cat([big[:, :col0].flatten(), big[:, col0 + n:].flatten()])
    assert bool((rest == -7.0).all())


@pytest.mark.parametrize("pad", [0, 8])
def test_gemm_bf16_output_larger_than_mall(pad):
    # A bf16 output of at least 256 MB (8192 x 16640: 272 MB) is written with
    # non-temporal stores (pad: rows ldy = N + pad apart, still 16-byte
    # aligned); the same product for the first 512 rows (17 MB, ordinary
    # stores) must give the same bits, every bf16 value must be RNE of the
    # FP32 output, and the padding columns must stay untouched.
    rng = np.random.default_rng(308)
    m, n, k = 8192, 16640, 256
    x, w = _xw(rng, m, n, k)
    offs = [0, 8192, n]
    aq = L.quantize_act(to_dev_bf16(x))
    pw = L.pack_weight(to_dev_bf16(w), offs)
    big = torch.full((m, n + pad), -7.0, dtype=torch.bfloat16, device="cuda")
    y16 = big[:, :n]
    L.gemm(aq, pw, out=y16)
    if pad:
        assert bool((big[:, n:] == -7.0).all())
    y32 = L.gemm(aq, pw, out_dtype=torch.float32)
    assert torch.equal(y16.view(torch.int16), y32.to(torch.bfloat16).view(torch.int16))
    del y32
    aq_top = L.quantize_act(to_dev_bf16(x[:512]), g=aq.g.item())    # the whole tensor's global scale
    y_top = L.gemm(aq_top, pw)
    torch.cuda.synchronize()
    assert torch.equal(y16[:512].view(torch.int16), y_top.view(torch.int16))
    rows = np.arange(0, m, 509)
    xp, xs, gx = OQ.quantize_tensor(x)
    wp, ws, gw = OQ.quantize_segments(w, offs)
    y_ref = OG.gemm_f64(xp, xs, gx, wp, ws, gw, offs, rows=rows)
    r_ref = OG.abs_bound(xp, xs, gx, wp, ws, gw, offs, rows=rows)
    got = y16[torch.from_numpy(rows).cuda()].float().cpu().numpy().astype(np.float64)
    # bf16 output: within the GEMM tolerance plus half a bf16 step
    err = np.abs(got - y_ref)
    assert (err <= 1e-4 * r_ref + np.abs(y_ref) * 2.0 ** -8 + 1e-30).all()


def test_gemm_segments_with_very_different_scales():
    rng = np.random.default_rng(301)
    k = 256
    x = bits_of(rng.standard_normal((96, k)))
    w = bits_of(np.concatenate([rng.standard_normal((64, k)) * 1e-4, rng.standard_normal((32, k)) * 30.0,
                                rng.standard_normal((160, k)) * 0.02]))
    check_small(x, w, [0, 64, 96, 256], what="segment scales")


def test_gemm_zero_activation_gives_zero():
    rng = np.random.default_rng(302)
    x = np.zeros((40, 64), dtype=np.uint16)
    w = bits_of(rng.standard_normal((64, 64)))
    y32, y16, aq, _ = run_gpu(x, w, [0, 64])
    assert aq.g.item() == 0.0
    assert torch.count_nonzero(y32).item() == 0


def test_gemm_is_deterministic_and_stays_in_bounds():
    rng = np.random.default_rng(303)
    x, w = _xw(rng, 200, 160, 512)
    aq = L.quantize_act(to_dev_bf16(x))
    pw = L.pack_weight(to_dev_bf16(w), [0, 100, 160])
    buf = torch.full((200 * 168 + 1024,), 12345.0, dtype=torch.float32, device="cuda")
    y = buf[: 200 * 168].view(200, 168)[:, :160]
    L.gemm(aq, pw, out=y)
    first = y.clone()
    for _ in range(3):
        L.gemm(aq, pw, out=y)
        assert torch.equal(y, first)
    torch.cuda.synchronize()
    pad = buf[: 200 * 168].view(200, 168)[:, 160:]
    assert torch.all(pad == 12345.0) and torch.all(buf[200 * 168:] == 12345.0)


def _sample_rows(m, tile):
    """Rows checked on a full workload: every row if m <= 32; else one row
    in every `tile`-row M-tile of the kernel (its position within the tile
    rotating with the tile index), all rows of the middle tile band, and the
    first and last 8 rows."""
    if m <= 32:
        return np.arange(m)
    tiles = (m + tile - 1) // tile
    rows = [t * tile + (t * 37 + 5) % tile for t in range(tiles)]
    mid = tiles // 2
    rows += list(range(mid * tile, min(m, (mid + 1) * tile)))
    rows += list(range(8)) + list(range(m - 8, m))
    return np.array(sorted(set(r for r in rows if r < m)))


@pytest.mark.parametrize("name", synth.CONFIG_ORDER + synth.DECODE_ORDER)
def test_gemm_full_workloads(name):
    wl = workload(name)
    cfg = wl["cfg"]
    log("%s: GEMM on GPU" % name)
    y32, y16, aq, pw = run_gpu(wl["x"], wl["w"], cfg.seg_offsets)
    assert np.float32(aq.g.item()) == wl["gx"]
    # BF16 output is the RNE of the FP32 output, everywhere.
    assert torch.equal(y16.contiguous().view(torch.int16), y32.to(torch.bfloat16).view(torch.int16))
    kernels = L.gemm_kernels(cfg.m, cfg.n, cfg.k)
    tile = 64 if "64x96" in kernels[0] else (32 if ("32x64" in kernels[0] or "32x32" in kernels[0]) else 256)
    rows = _sample_rows(cfg.m, tile)
    log("%s: oracle on %d rows (%d-row tiles: one per tile + a full band), kernels %s" % (
        name, len(rows), tile, kernels))
    args = (wl["xp"], wl["xs"], wl["gx"], wl["wp"], wl["ws"], wl["gw"], cfg.seg_offsets)
    y_ref = OG.gemm_f64(*args, rows=rows)
    r_ref = OG.abs_bound(*args, rows=rows)
    got = y32[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    rel = check_gemm(got, y_ref, r_ref, name)
    log("%s: relative Frobenius error %.3g" % (name, rel))
