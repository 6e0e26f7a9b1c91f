"""Block statistics at NVFP4 granularity (paper, Table 2 and its caption).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Used as sanity bands
for the synthetic inputs, never as parity pins.

* max/RMS: tensor maximum magnitude over the tensor RMS.
* kurtosis: E[x^4] / E[x^2]^2 over the tensor (3 for a Gaussian).
* one-hot blocks: share of 16-element blocks whose max/RMS exceeds 3.  Since
  a block holds 16 values, max^2 > 9 * mean(x^2) means one value carries more
  than 9/16 = 56.25% of the block energy (caption of Table 2); max/RMS of a
  block can never exceed sqrt(16) = 4 (section 2).
* relative quantization error: ||dq(q(x)) - x||_F / ||x||_F.
"""

import numpy as np

from .formats import bf16_bits_to_f64
from .quant import BLOCK, dequantize, quantize_tensor


def block_max_over_rms(x):
    """Per-block max|x| / RMS for a (rows, K) float array (NaN for all-zero
    blocks)."""
    rows, k = x.shape
    b = x.reshape(rows, k // BLOCK, BLOCK)
    rms = np.sqrt(np.mean(b * b, axis=2))
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.abs(b).max(axis=2) / rms


def tensor_stats(x_bits):
    x = bf16_bits_to_f64(x_bits)
    rms = np.sqrt(np.mean(x * x))
    m2 = np.mean(x ** 2)
    ratio = block_max_over_rms(x)
    valid = np.isfinite(ratio)
    packed, scales, g = quantize_tensor(x_bits)
    xq = dequantize(packed, scales, g)
    return {
        "max_over_rms": float(np.abs(x).max() / rms),
        "kurtosis": float(np.mean(x ** 4) / m2 ** 2),
        "one_hot_block_share": float(np.mean(ratio[valid] > 3.0)),
        "rel_quant_error": float(np.linalg.norm(xq - x) / np.linalg.norm(x)),
    }
