"""ctypes binding of libnvfp4.so (include/nvfp4.h).

Argument marshalling only: every computation runs in the HIP kernels behind
the C ABI.  PyTorch tensors serve as device buffers and the current PyTorch
stream as the HIP stream.  There is no fallback: if the library is missing,
loading raises.
"""

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnvfp4.so")

NVFP4_OK = 0
NVFP4_EINVAL = 1
NVFP4_EUNSUPPORTED = 2
NVFP4_EWORKSPACE = 3
NVFP4_EHIP = 4

NVFP4_DYNAMIC = 0
NVFP4_STATIC = 1
NVFP4_BF16 = 0
NVFP4_F32 = 1
NVFP4_BLOCK = 16
NVFP4_MAX_SEGMENTS = 8

# name -> (restype, argtypes), in the order of include/nvfp4.h
_c_int64, _vp, _sz, _int = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
SIGNATURES = {
    "nvfp4_status_str": (ctypes.c_char_p, [_int]),
    "nvfp4_last_hip_error": (_int, []),
    "nvfp4_quantize_act_workspace": (_sz, [_c_int64, _c_int64]),
    "nvfp4_quantize_act": (_int, [_vp, _c_int64, _c_int64, _c_int64, _vp, _vp, _vp, _int, _vp, _sz, _vp]),
    "nvfp4_quantize_act_noalloc": (_int, [_vp, _c_int64, _c_int64, _c_int64, _vp, _vp, _vp, _int, _vp]),
    "nvfp4_rmsnorm_quantize_act": (_int, [_vp, _c_int64, _c_int64, _c_int64, _vp, ctypes.c_float, _vp, _vp,
                                           _vp, _vp, _c_int64, _vp]),
    "nvfp4_packed_weight_bytes": (_sz, [_c_int64, _c_int64]),
    "nvfp4_pack_weight_workspace_bytes": (_sz, [_c_int64, _c_int64, _int]),
    "nvfp4_pack_weight": (_int, [_vp, _c_int64, _c_int64, _c_int64, _vp, _int, _vp, _int, _vp, _sz,
                                 _vp, _sz, _vp]),
    "nvfp4_unpack_weight": (_int, [_vp, _c_int64, _c_int64, _vp, _vp, _vp]),
    "nvfp4_harmonize_weight": (_int, [_vp, _c_int64, _c_int64, _vp, _int, _vp, _vp, _vp]),
    "nvfp4_gemm_workspace": (_sz, [_c_int64, _c_int64, _c_int64]),
    "nvfp4_gemm_with_workspace": (_int, [_vp, _vp, _vp, _c_int64, _c_int64, _vp, _c_int64, _vp, _int, _vp, _vp,
                                         _c_int64, _int, _vp, _sz, _vp]),
    "nvfp4_gemm_kernel": (ctypes.c_char_p, [_c_int64, _c_int64, _c_int64, _int, _int]),
    "nvfp4_gemm_gdn_gates": (_int, [_vp, _vp, _vp, _c_int64, _c_int64, _vp, _c_int64, _vp, _vp, _vp, _vp,
                                    _c_int64, _int, _vp]),
    "nvfp4_gemm": (_int, [_vp, _vp, _vp, _c_int64, _c_int64, _vp, _c_int64, _vp, _int, _vp, _vp,
                          _c_int64, _int, _vp]),
    "nvfp4_quantize_gemm_workspace": (_sz, [_c_int64, _c_int64, _c_int64]),
    "nvfp4_quantize_gemm": (_int, [_vp, _c_int64, _c_int64, _c_int64, _vp, _int, _vp, _sz, _vp, _c_int64,
                                   _vp, _int, _vp, _vp, _vp, _vp, _c_int64, _int, _vp]),
}

_lib = None


class Nvfp4Error(RuntimeError):
    def __init__(self, status, where):
        msg = lib().nvfp4_status_str(status).decode()
        if status == NVFP4_EHIP:
            msg += " (hipError %d)" % lib().nvfp4_last_hip_error()
        super().__init__("%s: %s" % (where, msg))
        self.status = status


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libnvfp4.so is not built (run python -m paper_2609_04098_amd.build_lib)")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(l, name)
            fn.restype, fn.argtypes = res, args
        _lib = l
    return _lib


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(getattr(stream, "cuda_stream", stream))
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(status, where):
    if status != NVFP4_OK:
        raise Nvfp4Error(status, where)


def _offsets(seg_offsets):
    arr = (ctypes.c_int64 * len(seg_offsets))(*[int(o) for o in seg_offsets])
    return arr, len(seg_offsets) - 1


def nvfp4_quantize_act_workspace(M, K):
    return lib().nvfp4_quantize_act_workspace(int(M), int(K))


def nvfp4_packed_weight_bytes(N, K):
    return lib().nvfp4_packed_weight_bytes(int(N), int(K))


def nvfp4_pack_weight_workspace_bytes(N, K, n_seg):
    return lib().nvfp4_pack_weight_workspace_bytes(int(N), int(K), int(n_seg))


def nvfp4_quantize_act(x, codes, scales, g_enc, mode=NVFP4_DYNAMIC, workspace=None, stream=None,
                       M=None, K=None, ldx=None):
    """x: bf16 [M, K] (row stride ldx); codes uint8 [M, K/2]; scales uint8
    [M, K/16]; g_enc float32 [1]; workspace uint8 of
    nvfp4_quantize_act_workspace bytes (dynamic mode)."""
    M = x.shape[0] if M is None else M
    K = x.shape[1] if K is None else K
    ldx = x.stride(0) if ldx is None else ldx
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib().nvfp4_quantize_act(_ptr(x), M, K, ldx, _ptr(codes), _ptr(scales), _ptr(g_enc), mode,
                                  _ptr(workspace), ws_bytes, _stream(stream))
    _check(st, "nvfp4_quantize_act")


def nvfp4_quantize_act_noalloc(x, codes, scales, g_enc, mode=NVFP4_DYNAMIC, stream=None, M=None, K=None, ldx=None):
    """nvfp4_quantize_act without a workspace (the library's per-device
    scratch holds the partial maxima); same layouts."""
    M = x.shape[0] if M is None else M
    K = x.shape[1] if K is None else K
    ldx = x.stride(0) if ldx is None else ldx
    st = lib().nvfp4_quantize_act_noalloc(_ptr(x), M, K, ldx, _ptr(codes), _ptr(scales), _ptr(g_enc), mode,
                                          _stream(stream))
    _check(st, "nvfp4_quantize_act_noalloc")


def nvfp4_rmsnorm_quantize_act(x, gamma, eps, codes, scales, g_enc, y=None, stream=None):
    """x bf16 [M, K] (row stride x.stride(0)); gamma bf16 [K]; g_enc float32
    [1] (the calibrated G); codes uint8 [M, K/2]; scales uint8 [M, K/16];
    y optional bf16 [M, K] output of the normalization."""
    M, K = x.shape
    ldy = 0 if y is None else y.stride(0)
    st = lib().nvfp4_rmsnorm_quantize_act(_ptr(x), M, K, x.stride(0), _ptr(gamma), float(eps), _ptr(codes),
                                          _ptr(scales), _ptr(g_enc), _ptr(y), ldy, _stream(stream))
    _check(st, "nvfp4_rmsnorm_quantize_act")


def nvfp4_pack_weight(w, seg_offsets, g_enc_seg, packed, mode=NVFP4_DYNAMIC, workspace=None,
                      stream=None):
    """w: bf16 [N, K]; seg_offsets: host list of n_seg + 1 ints; g_enc_seg
    float32 [n_seg]; packed uint8 of nvfp4_packed_weight_bytes(N, K) bytes."""
    offs, n_seg = _offsets(seg_offsets)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib().nvfp4_pack_weight(_ptr(w), w.shape[0], w.shape[1], w.stride(0), offs, n_seg,
                                 _ptr(g_enc_seg), mode, _ptr(packed), packed.numel(),
                                 _ptr(workspace), ws_bytes, _stream(stream))
    _check(st, "nvfp4_pack_weight")


def nvfp4_unpack_weight(packed, N, K, codes, scales, stream=None):
    st = lib().nvfp4_unpack_weight(_ptr(packed), N, K, _ptr(codes), _ptr(scales), _stream(stream))
    _check(st, "nvfp4_unpack_weight")


def nvfp4_harmonize_weight(packed, N, K, seg_offsets, g_enc_seg, g_shared, stream=None):
    """In place: one shared global scale for a fused weight group (written to
    g_shared, device float [1]), block scales re-rounded accordingly."""
    offs, n_seg = _offsets(seg_offsets)
    st = lib().nvfp4_harmonize_weight(_ptr(packed), N, K, offs, n_seg, _ptr(g_enc_seg), _ptr(g_shared),
                                      _stream(stream))
    _check(st, "nvfp4_harmonize_weight")


def nvfp4_gemm(a_codes, a_scales, a_g_enc, w_packed, N, seg_offsets, w_g_enc_seg, y,
               y_dtype=NVFP4_BF16, stream=None, M=None, K=None):
    """Y [M, N] (row stride y.stride(0)) = dq(A) dq(W)^T with per-segment
    global scales."""
    M = a_codes.shape[0] if M is None else M
    K = 2 * a_codes.shape[1] if K is None else K
    offs, n_seg = _offsets(seg_offsets)
    st = lib().nvfp4_gemm(_ptr(a_codes), _ptr(a_scales), _ptr(a_g_enc), M, K, _ptr(w_packed), N,
                          offs, n_seg, _ptr(w_g_enc_seg), _ptr(y), y.stride(0), y_dtype,
                          _stream(stream))
    _check(st, "nvfp4_gemm")


def nvfp4_gemm_workspace(M, N, K):
    return lib().nvfp4_gemm_workspace(int(M), int(N), int(K))


def nvfp4_gemm_with_workspace(a_codes, a_scales, a_g_enc, w_packed, N, seg_offsets, w_g_enc_seg, y,
                              y_dtype=NVFP4_BF16, workspace=None, stream=None, M=None, K=None):
    """nvfp4_gemm with a workspace (uint8 device tensor or None)."""
    M = a_codes.shape[0] if M is None else M
    K = 2 * a_codes.shape[1] if K is None else K
    offs, n_seg = _offsets(seg_offsets)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib().nvfp4_gemm_with_workspace(_ptr(a_codes), _ptr(a_scales), _ptr(a_g_enc), M, K, _ptr(w_packed), N,
                                         offs, n_seg, _ptr(w_g_enc_seg), _ptr(y), y.stride(0), y_dtype,
                                         _ptr(workspace), ws_bytes, _stream(stream))
    _check(st, "nvfp4_gemm_with_workspace")


def nvfp4_gemm_kernel(M, N, K, part=0, with_workspace=0):
    """Name of launch `part` of nvfp4_gemm (with_workspace 0) or of
    nvfp4_gemm_with_workspace (1) for this shape on the current device, or
    None."""
    r = lib().nvfp4_gemm_kernel(int(M), int(N), int(K), int(part), int(with_workspace))
    return None if r is None else r.decode()


def nvfp4_gemm_gdn_gates(a_codes, a_scales, a_g_enc, w_packed, H, w_g_enc_seg, a_log, dt_bias, y,
                         y_dtype=NVFP4_BF16, stream=None, M=None, K=None):
    """y [M, 2H] = (beta | alpha) of the fused b|a gate projection."""
    M = a_codes.shape[0] if M is None else M
    K = 2 * a_codes.shape[1] if K is None else K
    st = lib().nvfp4_gemm_gdn_gates(_ptr(a_codes), _ptr(a_scales), _ptr(a_g_enc), M, K, _ptr(w_packed), H,
                                    _ptr(w_g_enc_seg), _ptr(a_log), _ptr(dt_bias), _ptr(y), y.stride(0), y_dtype,
                                    _stream(stream))
    _check(st, "nvfp4_gemm_gdn_gates")


def nvfp4_quantize_gemm_workspace(M, N, K):
    return lib().nvfp4_quantize_gemm_workspace(int(M), int(N), int(K))


def nvfp4_quantize_gemm(x, a_g_enc, w_packed, N, seg_offsets, w_g_enc_seg, y, mode=NVFP4_DYNAMIC,
                        workspace=None, a_codes=None, a_scales=None, y_dtype=NVFP4_BF16, stream=None):
    """Y [M, N] = quantize(x) then the segment-scaled GEMM, fused (N <= 128 or
    M <= 32);
    x bf16 [M, K] (row stride x.stride(0)); optional a_codes / a_scales
    outputs."""
    M, K = x.shape
    offs, n_seg = _offsets(seg_offsets)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib().nvfp4_quantize_gemm(_ptr(x), M, K, x.stride(0), _ptr(a_g_enc), mode, _ptr(workspace), ws_bytes,
                                   _ptr(w_packed), N, offs, n_seg, _ptr(w_g_enc_seg), _ptr(a_codes),
                                   _ptr(a_scales), _ptr(y), y.stride(0), y_dtype, _stream(stream))
    _check(st, "nvfp4_quantize_gemm")
