"""NVFP4 W4A4 linear layer on top of the C ABI: buffer allocation and call
order only (the arithmetic is in the HIP kernels).

    pw = pack_weight(w, seg_offsets)          # offline: quantize + prepack W
    aq = quantize_act(x)                      # per call: codes, scales, G_A
    y  = gemm(aq, pw)                         # Y = dq(A) dq(W)^T, segment-scaled
"""

from dataclasses import dataclass
from typing import List

import torch

from . import nvfp4 as _c


@dataclass
class PackedWeight:
    packed: torch.Tensor          # uint8, GEMM-private layout
    g_seg: torch.Tensor           # float32 [n_seg], encode-direction global scales
    n: int
    k: int
    seg_offsets: List[int]


@dataclass
class QuantizedAct:
    codes: torch.Tensor           # uint8 [M, K/2]
    scales: torch.Tensor          # uint8 [M, K/16] (E4M3 codes)
    g: torch.Tensor               # float32 [1]
    m: int
    k: int


def _dev(t):
    return t.device


def pack_weight(w, seg_offsets=None, g_seg=None, stream=None) -> PackedWeight:
    """Quantize a bf16 [N, K] weight whose row ranges are separately
    calibrated segments; dynamic per-segment scales unless g_seg is given."""
    n, k = w.shape
    seg_offsets = [0, n] if seg_offsets is None else [int(o) for o in seg_offsets]
    n_seg = len(seg_offsets) - 1
    dev = _dev(w)
    packed = torch.empty(_c.nvfp4_packed_weight_bytes(n, k), dtype=torch.uint8, device=dev)
    if g_seg is None:
        gs = torch.empty(n_seg, dtype=torch.float32, device=dev)
        ws = torch.empty(_c.nvfp4_pack_weight_workspace_bytes(n, k, n_seg), dtype=torch.uint8, device=dev)
        _c.nvfp4_pack_weight(w, seg_offsets, gs, packed, _c.NVFP4_DYNAMIC, ws, stream)
    else:
        gs = torch.as_tensor(g_seg, dtype=torch.float32).to(dev).contiguous()
        _c.nvfp4_pack_weight(w, seg_offsets, gs, packed, _c.NVFP4_STATIC, None, stream)
    return PackedWeight(packed, gs, n, k, seg_offsets)


def unpack_weight(pw: PackedWeight, stream=None):
    """Canonical (codes uint8 [N, K/2], scales uint8 [N, K/16]) of a packed weight."""
    dev = pw.packed.device
    codes = torch.empty((pw.n, pw.k // 2), dtype=torch.uint8, device=dev)
    scales = torch.empty((pw.n, pw.k // 16), dtype=torch.uint8, device=dev)
    _c.nvfp4_unpack_weight(pw.packed, pw.n, pw.k, codes, scales, stream)
    return codes, scales


def harmonize_weight(pw: PackedWeight, in_place=False, stream=None) -> PackedWeight:
    """The one-global-scale form of a fused weight group (section 6 repair):
    a PackedWeight with a single segment whose scale is the shared G."""
    packed = pw.packed if in_place else pw.packed.clone()
    g = torch.empty(1, dtype=torch.float32, device=packed.device)
    _c.nvfp4_harmonize_weight(packed, pw.n, pw.k, pw.seg_offsets, pw.g_seg, g, stream)
    return PackedWeight(packed, g, pw.n, pw.k, [0, pw.n])


def alloc_act(m, k, device) -> QuantizedAct:
    return QuantizedAct(torch.empty((m, k // 2), dtype=torch.uint8, device=device),
                        torch.empty((m, k // 16), dtype=torch.uint8, device=device),
                        torch.empty(1, dtype=torch.float32, device=device), m, k)


def act_workspace(m, k, device):
    return torch.empty(_c.nvfp4_quantize_act_workspace(m, k), dtype=torch.uint8, device=device)


def quantize_act(x, g=None, out: QuantizedAct = None, workspace=None, stream=None) -> QuantizedAct:
    """Quantize a bf16 [M, K] activation (dynamic G unless ``g`` is given)."""
    m, k = x.shape
    dev = _dev(x)
    aq = alloc_act(m, k, dev) if out is None else out
    if g is None:
        ws = act_workspace(m, k, dev) if workspace is None else workspace
        _c.nvfp4_quantize_act(x, aq.codes, aq.scales, aq.g, _c.NVFP4_DYNAMIC, ws, stream)
    else:
        aq.g.copy_(torch.as_tensor([float(g)], dtype=torch.float32))
        _c.nvfp4_quantize_act(x, aq.codes, aq.scales, aq.g, _c.NVFP4_STATIC, None, stream)
    return aq


def rmsnorm_quantize_act(x, gamma, eps, g, out: QuantizedAct = None, y=None, stream=None) -> QuantizedAct:
    """RMSNorm of a bf16 [M, K] activation fused with its quantization under
    the calibrated global scale ``g`` (a float or a device float32 [1])."""
    m, k = x.shape
    aq = alloc_act(m, k, x.device) if out is None else out
    if torch.is_tensor(g):
        aq.g.copy_(g.reshape(1))
    else:
        aq.g.copy_(torch.as_tensor([float(g)], dtype=torch.float32))
    _c.nvfp4_rmsnorm_quantize_act(x, gamma, eps, aq.codes, aq.scales, aq.g, y, stream)
    return aq


def gemm_workspace(m, n, k, device):
    """Workspace for gemm() at this shape (None when the shape needs none)."""
    nbytes = _c.nvfp4_gemm_workspace(m, n, k)
    return None if nbytes == 0 else torch.empty(nbytes, dtype=torch.uint8, device=device)


def gemm(aq: QuantizedAct, pw: PackedWeight, out_dtype=torch.bfloat16, out=None, workspace=None, stream=None):
    """Y = dq(A) dq(W)^T through nvfp4_gemm_with_workspace (a workspace is
    allocated here when the shape uses one and none is given)."""
    if aq.k != pw.k:
        raise ValueError("K mismatch between activation and weight")
    dev = aq.codes.device
    y = out if out is not None else torch.empty((aq.m, pw.n), dtype=out_dtype, device=dev)
    kind = _c.NVFP4_F32 if y.dtype == torch.float32 else _c.NVFP4_BF16
    ws = gemm_workspace(aq.m, pw.n, aq.k, dev) if workspace is None else workspace
    _c.nvfp4_gemm_with_workspace(aq.codes, aq.scales, aq.g, pw.packed, pw.n, pw.seg_offsets, pw.g_seg, y, kind,
                                 ws, stream, M=aq.m, K=aq.k)
    return y


def gemm_no_workspace(aq: QuantizedAct, pw: PackedWeight, out_dtype=torch.bfloat16, out=None, stream=None):
    """The same product through nvfp4_gemm (no workspace)."""
    if aq.k != pw.k:
        raise ValueError("K mismatch between activation and weight")
    y = out if out is not None else torch.empty((aq.m, pw.n), dtype=out_dtype, device=aq.codes.device)
    kind = _c.NVFP4_F32 if y.dtype == torch.float32 else _c.NVFP4_BF16
    _c.nvfp4_gemm(aq.codes, aq.scales, aq.g, pw.packed, pw.n, pw.seg_offsets, pw.g_seg, y, kind,
                  stream, M=aq.m, K=aq.k)
    return y


def gemm_kernels(m, n, k, with_workspace=True):
    """Names of the kernels gemm() (or, with_workspace=False,
    gemm_no_workspace()) launches for an m x n x k call."""
    w = 1 if with_workspace else 0
    return [name for name in (_c.nvfp4_gemm_kernel(m, n, k, part, w) for part in (0, 1)) if name is not None]


def gemm_gdn_gates(aq: QuantizedAct, pw: PackedWeight, a_log, dt_bias, out_dtype=torch.bfloat16, out=None,
                   stream=None):
    """(beta | alpha) [M, 2H] from the fused [b; a] gate projection (Eq. 1)."""
    h = pw.n // 2
    if pw.seg_offsets != [0, h, 2 * h]:
        raise ValueError("the gate weight must be packed as two segments [b; a] of equal width")
    y = out if out is not None else torch.empty((aq.m, pw.n), dtype=out_dtype, device=aq.codes.device)
    kind = _c.NVFP4_F32 if y.dtype == torch.float32 else _c.NVFP4_BF16
    _c.nvfp4_gemm_gdn_gates(aq.codes, aq.scales, aq.g, pw.packed, h, pw.g_seg, a_log, dt_bias, y, kind, stream,
                            M=aq.m, K=aq.k)
    return y


def quantize_gemm_workspace(m, n, k, device):
    return torch.empty(_c.nvfp4_quantize_gemm_workspace(m, n, k), dtype=torch.uint8, device=device)


def quantize_gemm(x, pw: PackedWeight, g=None, out_dtype=torch.bfloat16, out=None, act_out: QuantizedAct = None,
                  workspace=None, stream=None):
    """Act-quant fused into the GEMM (N <= 128, or M <= 32): y [M, N] equal to
    gemm(quantize_act(x, g), pw).  Dynamic G unless ``g`` is given; the
    activation codes/scales/G are written to ``act_out`` when it is given.
    Returns (y, G as a device float32 [1])."""
    m, k = x.shape
    if k != pw.k:
        raise ValueError("K mismatch between activation and weight")
    dev = _dev(x)
    y = out if out is not None else torch.empty((m, pw.n), dtype=out_dtype, device=dev)
    kind = _c.NVFP4_F32 if y.dtype == torch.float32 else _c.NVFP4_BF16
    gbuf = act_out.g if act_out is not None else torch.empty(1, dtype=torch.float32, device=dev)
    codes = act_out.codes if act_out is not None else None
    scales = act_out.scales if act_out is not None else None
    ws = quantize_gemm_workspace(m, pw.n, k, dev) if workspace is None else workspace
    if g is None:
        _c.nvfp4_quantize_gemm(x, gbuf, pw.packed, pw.n, pw.seg_offsets, pw.g_seg, y, _c.NVFP4_DYNAMIC, ws,
                               codes, scales, kind, stream)
    else:
        gbuf.copy_(torch.as_tensor([float(g)], dtype=torch.float32))
        _c.nvfp4_quantize_gemm(x, gbuf, pw.packed, pw.n, pw.seg_offsets, pw.g_seg, y, _c.NVFP4_STATIC, ws,
                               codes, scales, kind, stream)
    return y, gbuf


def linear(x, pw: PackedWeight, out_dtype=torch.bfloat16):
    """y = x W^T through NVFP4 W4A4: dynamic act-quant, then the GEMM."""
    return gemm(quantize_act(x), pw, out_dtype)
