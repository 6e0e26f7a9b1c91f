"""Seeded synthetic inputs for the NVFP4 W4A4 linear layer.

This module holds no quantization or GEMM arithmetic; it only draws inputs.
Both the HIP path and the CPU oracle consume the exact bf16 bytes produced
here.

Stand-ins for the paper's workloads (the residual stream of a 27B hybrid
model with hidden size 5120, section 2; its statistics in section 5.1 and
Table 2: heavy per-channel outliers, max/RMS in the tens to hundreds, 5-32% of
16-element blocks dominated by one value).  The real activations, weights and
evaluation data are not available, so every tensor is synthetic:

* residual-stream activations: N(0, 1) with a seeded 0.5% of channels scaled
  by a per-channel factor drawn from U(50, 200);
* heavy-tailed activations (input of the MLP down projection): Student-t with
  3 degrees of freedom, times 0.5;
* weights: N(0, sigma) per fused segment, with the segment's own sigma.

Recipe: numpy ``Generator(PCG64(SeedSequence([seed, config, tensor])))``;
samples are drawn in float64, rounded to float32 (round to nearest even),
then rounded to bf16 (round to nearest even on the bit pattern).  Rows are
drawn in order in chunks, which gives the same stream as one draw.
"""

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np


@dataclass(frozen=True)
class Config:
    name: str
    index: int
    m: int
    k: int
    segments: Tuple[int, ...]            # output width of each fused segment
    seg_sigma: Tuple[float, ...]         # weight std of each segment
    x_kind: str                          # "normal_channels", "residual", "student_t"
    outlier_channels: Tuple[int, ...] = ()   # fixed outlier channels (tiny case)
    outlier_factor: float = 100.0
    description: str = ""

    @property
    def n(self):
        return int(sum(self.segments))

    @property
    def seg_offsets(self):
        return [0] + list(np.cumsum(self.segments).astype(int))

    @property
    def flops(self):
        return 2.0 * self.m * self.n * self.k


CONFIGS = {
    "tiny": Config(
        "tiny", 0, 64, 256, (128,), (0.02,), "normal_channels",
        outlier_channels=(3, 100), outlier_factor=100.0,
        description="tiny NVFP4 W4A4 linear 64x128x256, 2 outlier channels x100"),
    "gdn_qkv": Config(
        "gdn_qkv", 1, 4096, 5120, (2048, 2048, 4096),
        (0.02 * 1.0, 0.02 * 1.5, 0.02 * 0.7), "residual",
        description="fused GDN q/k/v input projection at prefill, 4096x8192x5120"),
    "mlp_gate_up": Config(
        "mlp_gate_up", 2, 8192, 5120, (17408, 17408),
        (0.015 * 1.0, 0.015 * 1.3), "residual",
        description="fused MLP gate/up projection, 8192x34816x5120"),
    "mlp_down": Config(
        "mlp_down", 3, 8192, 17408, (5120,), (0.01,), "student_t",
        description="MLP down projection, Student-t(3) inputs, 8192x5120x17408"),
    "ab_gates": Config(
        "ab_gates", 4, 32768, 5120, (48, 48), (0.05, 0.05), "residual",
        description="tall-skinny GDN a/b gate projection, 32768x96x5120"),
    # Decode-shaped calls of the gate/up projection: a batch of 1 or 32
    # tokens against the full fused weight (weight-bandwidth-bound).
    "decode_m32": Config(
        "decode_m32", 5, 32, 5120, (17408, 17408),
        (0.015 * 1.0, 0.015 * 1.3), "residual",
        description="decode-shape gate/up projection, 32 tokens, 32x34816x5120"),
    "decode_m1": Config(
        "decode_m1", 6, 1, 5120, (17408, 17408),
        (0.015 * 1.0, 0.015 * 1.3), "residual",
        description="decode-shape gate/up projection, 1 token, 1x34816x5120"),
}

CONFIG_ORDER = ["tiny", "gdn_qkv", "mlp_gate_up", "mlp_down", "ab_gates"]
DECODE_ORDER = ["decode_m32", "decode_m1"]

TENSOR_X = 0
TENSOR_W = 1


def rng_for(seed, config_index, tensor):
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([int(seed), int(config_index), int(tensor)])))


def f64_to_bf16_bits(a):
    """float64 -> float32 (RNE) -> bf16 bit pattern (RNE), as uint16.
    Inputs are finite."""
    f32 = np.asarray(a, dtype=np.float64).astype(np.float32)
    u = f32.view(np.uint32).astype(np.uint64)
    rounded = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def make_x(cfg: Config, seed=0, rows=None, chunk=1024):
    """Activation tensor (rows, K) as bf16 bit patterns (uint16).  ``rows``
    limits the draw to the first rows of the full tensor (same values)."""
    rows = cfg.m if rows is None else int(rows)
    rng = rng_for(seed, cfg.index, TENSOR_X)
    k = cfg.k
    # Channel scaling is drawn first so that it does not depend on ``rows``.
    factor = np.ones(k, dtype=np.float64)
    if cfg.x_kind == "normal_channels":
        factor[list(cfg.outlier_channels)] = cfg.outlier_factor
    elif cfg.x_kind == "residual":
        n_hot = int(round(0.005 * k))
        hot = rng.choice(k, size=n_hot, replace=False)
        factor[hot] = rng.uniform(50.0, 200.0, size=n_hot)
    out = np.empty((rows, k), dtype=np.uint16)
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        if cfg.x_kind == "student_t":
            v = rng.standard_t(3.0, size=(r1 - r0, k)) * 0.5
        else:
            v = rng.standard_normal(size=(r1 - r0, k)) * factor[None, :]
        out[r0:r1] = f64_to_bf16_bits(v)
    return out


def make_w(cfg: Config, seed=0, chunk=1024):
    """Fused weight (N, K) as bf16 bit patterns; segment s has rows
    [seg_offsets[s], seg_offsets[s+1]) drawn N(0, seg_sigma[s])."""
    rng = rng_for(seed, cfg.index, TENSOR_W)
    out = np.empty((cfg.n, cfg.k), dtype=np.uint16)
    offs = cfg.seg_offsets
    for s in range(len(cfg.segments)):
        for r0 in range(offs[s], offs[s + 1], chunk):
            r1 = min(offs[s + 1], r0 + chunk)
            v = rng.standard_normal(size=(r1 - r0, cfg.k)) * cfg.seg_sigma[s]
            out[r0:r1] = f64_to_bf16_bits(v)
    return out
