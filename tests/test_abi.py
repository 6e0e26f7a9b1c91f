"""The C-ABI library loads, exports every function include/nvfp4.h declares,
and rejects invalid arguments synchronously, before any HIP call (these paths
need no GPU)."""

import ctypes
import os
import re

import pytest

from paper_2609_04098_amd import nvfp4 as C

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nvfp4.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nvfp4_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ["nvfp4_quantize_act", "nvfp4_pack_weight", "nvfp4_gemm", "nvfp4_unpack_weight"]:
        assert n in names
    assert set(names) == set(C.SIGNATURES)


def test_library_exports_every_declared_symbol():
    lib = C.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings():
    lib = C.lib()
    for s in range(5):
        assert lib.nvfp4_status_str(s).decode().startswith("NVFP4")
    assert lib.nvfp4_last_hip_error() == 0


def test_sizes():
    lib = C.lib()
    assert lib.nvfp4_quantize_act_workspace(8192, 5120) >= 4
    # N padded to 32, K to 64: codes Np*Kp/2 + scales Np*Kp/16
    assert lib.nvfp4_packed_weight_bytes(96, 5120) == 96 * 5120 // 2 + 96 * 5120 // 16
    assert lib.nvfp4_packed_weight_bytes(100, 80) == 128 * 128 // 2 + 128 * 128 // 16
    assert lib.nvfp4_packed_weight_bytes(0, 80) == 0
    assert lib.nvfp4_pack_weight_workspace_bytes(10, 32, 3) >= 3 * 4


FAKE = 0x100000   # 16-byte aligned, never dereferenced: validation fails first


def _offs(lst):
    return (ctypes.c_int64 * len(lst))(*lst)


def test_quantize_act_rejects_bad_arguments():
    f = C.lib().nvfp4_quantize_act
    ws = C.lib().nvfp4_quantize_act_workspace(4, 32)
    ok = dict(x=FAKE, M=4, K=32, ldx=32, codes=FAKE, scales=FAKE, g=FAKE, mode=0, ws=FAKE, wsb=ws)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["x"], a["M"], a["K"], a["ldx"], a["codes"], a["scales"], a["g"], a["mode"],
                 a["ws"], a["wsb"], None)
    assert call(K=24) == C.NVFP4_EINVAL             # K % 16 != 0
    assert call(M=-1) == C.NVFP4_EINVAL
    assert call(ldx=16) == C.NVFP4_EINVAL           # ldx < K
    assert call(ldx=36) == C.NVFP4_EINVAL           # ldx % 8 != 0
    assert call(x=None) == C.NVFP4_EINVAL
    assert call(codes=FAKE + 4) == C.NVFP4_EINVAL   # misaligned
    assert call(g=None) == C.NVFP4_EINVAL
    assert call(mode=7) == C.NVFP4_EINVAL
    assert call(ws=None) == C.NVFP4_EINVAL
    assert call(wsb=ws - 1) == C.NVFP4_EWORKSPACE
    assert call(M=1 << 20, K=1 << 12, ldx=1 << 12) == C.NVFP4_EINVAL   # M*K >= 2^31


def test_pack_weight_rejects_bad_arguments():
    f = C.lib().nvfp4_pack_weight
    n, k = 64, 256
    pb = C.lib().nvfp4_packed_weight_bytes(n, k)
    wsb = C.lib().nvfp4_pack_weight_workspace_bytes(n, k, 2)

    def call(offs=(0, 32, 64), n_seg=2, N=n, K=k, ldw=k, packed_bytes=pb, ws=FAKE, mode=0, g=FAKE):
        return f(FAKE, N, K, ldw, _offs(list(offs)), n_seg, g, mode, FAKE, packed_bytes, ws, wsb, None)
    assert call(offs=(0, 32, 32), n_seg=2) == C.NVFP4_EINVAL       # not strictly increasing
    assert call(offs=(0, 32, 60), n_seg=2) == C.NVFP4_EINVAL       # does not end at N
    assert call(offs=(1, 32, 64), n_seg=2) == C.NVFP4_EINVAL       # does not start at 0
    assert call(offs=tuple(range(0, 72, 8)), n_seg=9, N=64) == C.NVFP4_EINVAL  # > 8 segments
    assert call(n_seg=0) == C.NVFP4_EINVAL
    assert call(K=8, ldw=8) == C.NVFP4_EINVAL
    assert call(packed_bytes=pb - 1) == C.NVFP4_EWORKSPACE
    assert call(ws=None) == C.NVFP4_EINVAL
    assert call(g=None) == C.NVFP4_EINVAL
    assert f(FAKE, n, k, k, None, 1, FAKE, 0, FAKE, pb, FAKE, wsb, None) == C.NVFP4_EINVAL


def test_gemm_rejects_bad_arguments():
    f = C.lib().nvfp4_gemm

    def call(M=16, K=64, N=32, offs=(0, 32), n_seg=1, ldy=32, dtype=0, y=FAKE, a=FAKE, wg=FAKE):
        return f(a, FAKE, FAKE, M, K, FAKE, N, _offs(list(offs)), n_seg, wg, y, ldy, dtype, None)
    assert call(K=40) == C.NVFP4_EINVAL
    assert call(K=0) == C.NVFP4_EINVAL
    assert call(N=0, offs=(0, 0)) == C.NVFP4_EINVAL
    assert call(ldy=24) == C.NVFP4_EINVAL
    assert call(y=FAKE + 2, dtype=1) == C.NVFP4_EINVAL     # f32 output not 4-byte aligned
    assert call(dtype=5) == C.NVFP4_EINVAL
    assert call(offs=(0, 16, 32), n_seg=1) == C.NVFP4_EINVAL
    assert call(y=None) == C.NVFP4_EINVAL
    assert call(a=FAKE + 8) == C.NVFP4_EINVAL
    assert call(wg=None) == C.NVFP4_EINVAL
    assert f(FAKE, FAKE, FAKE, 16, 64, FAKE, 32, None, 1, FAKE, FAKE, 32, 0, None) == C.NVFP4_EINVAL


def test_gemm_with_workspace_rejects_bad_arguments():
    f = C.lib().nvfp4_gemm_with_workspace

    def call(M=16, K=64, N=32, offs=(0, 32), n_seg=1, ldy=32, dtype=0, y=FAKE, ws=None, wsb=0):
        return f(FAKE, FAKE, FAKE, M, K, FAKE, N, _offs(list(offs)), n_seg, FAKE, y, ldy, dtype, ws, wsb, None)
    assert call(K=40) == C.NVFP4_EINVAL                     # the nvfp4_gemm checks come first
    assert call(ldy=24) == C.NVFP4_EINVAL
    assert call(y=None) == C.NVFP4_EINVAL
    assert call(ws=FAKE + 8, wsb=1 << 20) == C.NVFP4_EINVAL  # misaligned workspace
    # sizes: no device here (or a shape with full rounds): 0
    assert C.lib().nvfp4_gemm_workspace(16, 32, 40) == 0     # invalid K
    assert C.lib().nvfp4_gemm_workspace(-1, 32, 64) == 0


def test_unpack_rejects_bad_arguments():
    f = C.lib().nvfp4_unpack_weight
    assert f(FAKE, 0, 32, FAKE, FAKE, None) == C.NVFP4_EINVAL
    assert f(FAKE, 8, 24, FAKE, FAKE, None) == C.NVFP4_EINVAL
    assert f(None, 8, 32, FAKE, FAKE, None) == C.NVFP4_EINVAL


def test_harmonize_rejects_bad_arguments():
    f = C.lib().nvfp4_harmonize_weight

    def call(N=32, K=64, offs=(0, 16, 32), n_seg=2, packed=FAKE, g=FAKE, gs=FAKE + 64):
        return f(packed, N, K, _offs(list(offs)), n_seg, g, gs, None)
    assert call(K=40) == C.NVFP4_EINVAL
    assert call(N=0, offs=(0, 0), n_seg=1) == C.NVFP4_EINVAL
    assert call(offs=(0, 16, 16)) == C.NVFP4_EINVAL
    assert call(offs=(0, 16, 30)) == C.NVFP4_EINVAL
    assert call(packed=None) == C.NVFP4_EINVAL
    assert call(packed=FAKE + 4) == C.NVFP4_EINVAL
    assert call(g=None) == C.NVFP4_EINVAL
    assert call(gs=None) == C.NVFP4_EINVAL
    assert call(gs=FAKE + 4) == C.NVFP4_EINVAL            # g_shared inside g_enc_seg
    assert call(gs=FAKE + 66) == C.NVFP4_EINVAL           # misaligned


def test_library_has_no_unresolved_own_symbols():
    """Every kernel the launchers reference is defined in the library (a
    kernel template whose host stub is not emitted shows up as an undefined
    symbol only when the library is loaded with lazy binding)."""
    import subprocess
    out = subprocess.run(["nm", "-D", "--undefined-only", C.LIB_PATH], capture_output=True, text=True)
    assert out.returncode == 0
    own = [l for l in out.stdout.splitlines() if "nvfp4" in l]
    assert not own, own


def test_rmsnorm_quantize_rejects_bad_arguments():
    f = C.lib().nvfp4_rmsnorm_quantize_act

    def call(M=8, K=64, ldx=64, gamma=FAKE, eps=1e-6, codes=FAKE, g=FAKE, y=None, ldy=0, x=FAKE):
        return f(x, M, K, ldx, gamma, eps, codes, FAKE, g, y, ldy, None)
    assert call(K=40) == C.NVFP4_EINVAL
    assert call(K=0) == C.NVFP4_EINVAL
    assert call(ldx=32) == C.NVFP4_EINVAL
    assert call(eps=-1.0) == C.NVFP4_EINVAL
    assert call(eps=float("inf")) == C.NVFP4_EINVAL
    assert call(eps=float("nan")) == C.NVFP4_EINVAL
    assert call(gamma=None) == C.NVFP4_EINVAL
    assert call(gamma=FAKE + 8) == C.NVFP4_EINVAL
    assert call(g=None) == C.NVFP4_EINVAL
    assert call(codes=None) == C.NVFP4_EINVAL
    assert call(y=FAKE, ldy=32) == C.NVFP4_EINVAL
    assert call(y=FAKE + 8, ldy=64) == C.NVFP4_EINVAL
    assert call(x=FAKE + 2) == C.NVFP4_EINVAL


def test_gdn_gates_rejects_bad_arguments():
    f = C.lib().nvfp4_gemm_gdn_gates

    def call(M=16, K=128, H=48, ldy=96, dtype=0, alog=FAKE, dt=FAKE, y=FAKE, a=FAKE):
        return f(a, FAKE, FAKE, M, K, FAKE, H, FAKE, alog, dt, y, ldy, dtype, None)
    assert call(H=0) == C.NVFP4_EINVAL
    assert call(ldy=95) == C.NVFP4_EINVAL
    assert call(alog=None) == C.NVFP4_EINVAL
    assert call(dt=FAKE + 2) == C.NVFP4_EINVAL
    assert call(y=None) == C.NVFP4_EINVAL
    assert call(dtype=3) == C.NVFP4_EINVAL
    assert call(K=80) == C.NVFP4_EUNSUPPORTED       # the gate epilogue needs K % 64 == 0


def test_quantize_gemm_rejects_bad_arguments():
    f = C.lib().nvfp4_quantize_gemm
    offs = _offs([0, 48, 96])

    def call(M=16, K=128, ldx=128, mode=C.NVFP4_STATIC, ws=None, wsb=0, N=96, segs=offs, nseg=2, codes=None,
             scales=None, y=FAKE, ldy=96, dtype=0, x=FAKE, g=FAKE):
        return f(x, M, K, ldx, g, mode, ws, wsb, FAKE, N, segs, nseg, FAKE, codes, scales, y, ldy, dtype, None)
    assert call(mode=5) == C.NVFP4_EINVAL
    assert call(K=40) == C.NVFP4_EINVAL              # K % 16 != 0
    assert call(ldx=120) == C.NVFP4_EINVAL           # ldx < K
    assert call(ldx=132) == C.NVFP4_EINVAL           # ldx % 8 != 0
    assert call(x=FAKE + 8) == C.NVFP4_EINVAL        # x not 16-byte aligned
    assert call(g=None) == C.NVFP4_EINVAL
    assert call(codes=FAKE) == C.NVFP4_EINVAL        # codes without scales
    assert call(codes=FAKE + 4, scales=FAKE) == C.NVFP4_EINVAL
    assert call(ldy=95) == C.NVFP4_EINVAL
    assert call(segs=_offs([0, 48, 96, 120]), nseg=3) == C.NVFP4_EINVAL   # table ends past N
    assert call(y=FAKE + 1) == C.NVFP4_EINVAL
    assert call(mode=C.NVFP4_DYNAMIC) == C.NVFP4_EINVAL          # no workspace
    assert call(mode=C.NVFP4_DYNAMIC, ws=FAKE, wsb=4) == C.NVFP4_EWORKSPACE
    assert call(M=33, N=160, segs=_offs([0, 160]), nseg=1, ldy=160) == C.NVFP4_EUNSUPPORTED   # N > 128, M > 32
    # M <= 32 with N > 128 (the decode path) needs a workspace in both modes
    assert call(M=32, N=160, segs=_offs([0, 160]), nseg=1, ldy=160) == C.NVFP4_EINVAL
    wsb = C.lib().nvfp4_quantize_gemm_workspace(32, 160, 128)
    assert wsb >= 4096 + 32 * 128 // 2 + 32 * 128 // 16
    assert call(M=32, N=160, segs=_offs([0, 160]), nseg=1, ldy=160, ws=FAKE, wsb=wsb - 1) == C.NVFP4_EWORKSPACE
    assert call(K=80, ldx=80) == C.NVFP4_EUNSUPPORTED             # K % 64 != 0


def _no_gpu():
    try:
        import torch
        return not torch.cuda.is_available()
    except Exception:
        return True


@pytest.mark.skipif(not _no_gpu(), reason="runs where there is no GPU: valid arguments stop at the device check")
def test_valid_arguments_stop_at_the_device_check():
    lib = C.lib()
    ws = lib.nvfp4_quantize_act_workspace(64, 256)
    offs = _offs([0, 48, 96])
    calls = [
        lambda: lib.nvfp4_quantize_act(FAKE, 64, 256, 256, FAKE, FAKE, FAKE, C.NVFP4_DYNAMIC, FAKE, ws, None),
        lambda: lib.nvfp4_quantize_act_noalloc(FAKE, 64, 256, 256, FAKE, FAKE, FAKE, C.NVFP4_DYNAMIC, None),
        lambda: lib.nvfp4_rmsnorm_quantize_act(FAKE, 64, 256, 256, FAKE, 1e-6, FAKE, FAKE, FAKE, None, 0, None),
        lambda: lib.nvfp4_pack_weight(FAKE, 96, 256, 256, offs, 2, FAKE, C.NVFP4_STATIC,
                                      FAKE, lib.nvfp4_packed_weight_bytes(96, 256), None, 0, None),
        lambda: lib.nvfp4_unpack_weight(FAKE, 96, 256, FAKE, FAKE, None),
        lambda: lib.nvfp4_harmonize_weight(FAKE, 96, 256, offs, 2, FAKE, FAKE + 64, None),
        lambda: lib.nvfp4_gemm(FAKE, FAKE, FAKE, 64, 256, FAKE, 96, offs, 2, FAKE, FAKE, 96, C.NVFP4_BF16, None),
        lambda: lib.nvfp4_gemm_with_workspace(FAKE, FAKE, FAKE, 64, 256, FAKE, 96, offs, 2, FAKE, FAKE, 96,
                                              C.NVFP4_BF16, None, 0, None),
        lambda: lib.nvfp4_gemm_gdn_gates(FAKE, FAKE, FAKE, 64, 256, FAKE, 48, FAKE, FAKE, FAKE, FAKE, 96,
                                         C.NVFP4_F32, None),
        lambda: lib.nvfp4_quantize_gemm(FAKE, 64, 256, 256, FAKE, C.NVFP4_STATIC, None, 0, FAKE, 96, offs, 2, FAKE,
                                        None, None, FAKE, 96, C.NVFP4_BF16, None),
    ]
    for call in calls:
        assert call() in (C.NVFP4_EHIP, C.NVFP4_EUNSUPPORTED)
    assert lib.nvfp4_gemm_kernel(8192, 34816, 5120, 0, 0) is None
    assert lib.nvfp4_gemm_kernel(8192, 34816, 5120, 2, 0) is None
    assert lib.nvfp4_gemm_kernel(8192, 5120, 17408, 1, 1) is None
    assert lib.nvfp4_gemm_workspace(8192, 5120, 17408) == 0


def test_quantize_act_noalloc_rejects_bad_arguments():
    f = C.lib().nvfp4_quantize_act_noalloc

    def call(x=FAKE, M=4, K=32, ldx=32, codes=FAKE, scales=FAKE, g=FAKE, mode=0):
        return f(x, M, K, ldx, codes, scales, g, mode, None)
    assert call(K=24) == C.NVFP4_EINVAL
    assert call(M=-1) == C.NVFP4_EINVAL
    assert call(ldx=16) == C.NVFP4_EINVAL
    assert call(x=None) == C.NVFP4_EINVAL
    assert call(scales=FAKE + 4) == C.NVFP4_EINVAL
    assert call(g=None) == C.NVFP4_EINVAL
    assert call(mode=2) == C.NVFP4_EINVAL
    assert call(M=1 << 20, K=1 << 12, ldx=1 << 12) == C.NVFP4_EINVAL
    # The scratch (4096 bytes per device) covers every shape's workspace.
    for m, k in [(1, 16), (8192, 5120), (32768, 5120), (131071, 16384)]:
        assert C.lib().nvfp4_quantize_act_workspace(m, k) <= 4096
