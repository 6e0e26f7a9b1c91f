"""CPU oracle for the NVFP4 W4A4 linear layer.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, table or
constant generator with the HIP kernels under ``paper_2609_04098_amd/csrc``.

What it computes (paper, section 2 "NVFP4"; section 6 "Per-module calibration
vs. fused-GEMM scaling"):

* ``formats``  E2M1 element values, OCP E4M3FN block-scale values, bf16 decode,
  and exact round-to-nearest-even onto a value grid.
* ``quant``    the per-tensor FP32 global scale, the per-16-element E4M3 block
  scale (block max / 6 under the global scale), E2M1 encoding, nibble packing,
  and dequantization ("fake quantization": quantize, dequantize, continue in
  high precision, section 5 introduction).
* ``gemm``     the dequantized GEMM Y = dq(A) dq(W)^T in FP64 with each fused
  output segment scaled by its own global scales (the per-module scales of
  section 6), an exact int64 form of the same sum, and the sum of |a_k b_k|
  used by the tolerance.
* ``harmonize`` the repair of section 6 for a fused weight group: one shared
  global scale with the ratio folded into re-rounded E4M3 block scales.
* ``gates``    the GDN gate transform (Eq. 1) of the fused a/b projection.
* ``norm``     RMSNorm in front of the quantizer (for the one-pass
  normalize-and-quantize path with a calibrated activation scale).
* ``stats``    block statistics of Table 2 (max/RMS, kurtosis, one-hot blocks,
  relative quantization error), used only as sanity bands for synthetic data.

Every floating-point decision is taken in exact arithmetic (float64 holds
every product that is compared, see ``quant``), so codes and scales are a
function of the inputs alone, independent of any operation order.
"""

from . import formats, gates, quant, gemm, harmonize, norm, stats  # noqa: F401
