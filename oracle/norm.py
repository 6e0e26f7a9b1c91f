"""RMS normalization in front of the activation quantizer (the step before
the W4A4 linear layer).  The paper serves its W4A4 model with activation
scales calibrated offline (section 3, "Checkpoints"); with a fixed
(static) global scale the normalization and the quantization can be done in
one pass over the activations.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Reading (the paper names the norm but not its formula): the usual RMSNorm,
y = x / sqrt(mean_k(x^2) + eps) * gamma per row, evaluated in float64 and
rounded once to bf16 (round to nearest even); the quantizer then takes those
bf16 values with the given global scale.
"""

import numpy as np

from .formats import bf16_bits_to_f64, f64_to_bf16_bits


def rmsnorm_f64(x_bits, gamma_bits, eps):
    """y in float64 (rows, K) for bf16 inputs x (rows, K) and gamma (K,)."""
    x = bf16_bits_to_f64(x_bits)
    g = bf16_bits_to_f64(gamma_bits)
    ms = np.mean(x * x, axis=1)
    return x / np.sqrt(ms + float(np.float32(eps)))[:, None] * g[None, :]


def rmsnorm_bf16(x_bits, gamma_bits, eps):
    """bf16 bit patterns of RMSNorm(x) (one rounding of the float64 value)."""
    return f64_to_bf16_bits(rmsnorm_f64(x_bits, gamma_bits, eps))
