"""Seeded synthetic inputs for the few-bit activation path.

The paper's workloads (GLUE fine-tuning, ImageNet ResNets, ruDALL-E) need
datasets and trained weights; these tensors stand in for the activation
inputs and incoming gradients of such models, with the shapes of a BERT-base
FFN intermediate, a ResNet stage, a large-LM FFN and two long odd-length
vectors.

This module holds no arithmetic of the method: it only draws random numbers
and rounds them to the storage type.  Both the oracle-side tests and the GPU
path consume exactly these bit patterns.

Recipe (all draws in float64 with numpy's PCG64 ``default_rng``):
  * each workload has its own seed s (0 .. 4 below): x is drawn with seed
    s, grad_out with seed s + 1000;
  * N(mu, var) names the variance: N(0, 1e-2) has sigma 0.1;
  * "1% outliers": an i.i.d. Bernoulli(0.01) mask (uniform draws from seed
    s + 2000) replaces z by 10 z;
  * float64 -> float32 by numpy (round to nearest even); bf16 from that
    float32 by torch's CPU conversion (round to nearest even); fp16 from the
    float64 by numpy (round to nearest even);
  * arrays are generated in chunks of 2^24 elements from one stream, which
    yields the same values as a single draw.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

CHUNK = 1 << 24


@dataclass(frozen=True)
class Workload:
    name: str
    act: str                 # gelu | silu | sigmoid | tanh
    bits: tuple              # bit widths run on this input
    dtype: str               # f32 | f16 | bf16
    shape: tuple
    x_dist: str              # normal | mixture | uniform
    x_scale: float           # sigma (normal / mixture core) or half-width (uniform)
    g_sigma: float
    seed: int
    fit: dict = field(default_factory=dict)   # weight used for the table fit

    @property
    def n(self) -> int:
        n = 1
        for d in self.shape:
            n *= d
        return n


WORKLOADS = {
    "gelu3_f32_1m": Workload(
        "gelu3_f32_1m", "gelu", (3,), "f32", (1048576,), "normal", 1.0, 1.0, 0,
        {"kind": "normal", "A": -10.0, "B": 10.0, "sigma": 1.0, "n_grid": 4000}),
    "gelu3_bf16_bert_ffn_8x512x3072": Workload(
        "gelu3_bf16_bert_ffn_8x512x3072", "gelu", (3,), "bf16", (8, 512, 3072), "normal", 1.5,
        0.1, 1,
        {"kind": "normal", "A": -15.0, "B": 15.0, "sigma": 1.5, "n_grid": 6000}),
    "silu2_f16_resnet_64x256x56x56": Workload(
        "silu2_f16_resnet_64x256x56x56", "silu", (2,), "f16", (64, 256, 56, 56), "normal", 1.0,
        1.0, 2,
        {"kind": "normal", "A": -10.0, "B": 10.0, "sigma": 1.0, "n_grid": 4000}),
    "gelu_bf16_lm_ffn_16x2048x8192": Workload(
        "gelu_bf16_lm_ffn_16x2048x8192", "gelu", (1, 2, 3, 4), "bf16", (16, 2048, 8192), "mixture",
        1.0, 1.0, 3,
        {"kind": "mixture", "A": -40.0, "B": 40.0, "sigma": 1.0, "p": 0.01,
         "sigma2": 10.0, "n_grid": 8000}),
    "sigmoid4_f32_odd_67108863": Workload(
        "sigmoid4_f32_odd_67108863", "sigmoid", (4,), "f32", (67108863,), "uniform", 8.0, 1.0, 4,
        {"kind": "uniform", "A": -8.0, "B": 8.0, "n_grid": 3200}),
    "tanh3_f32_odd_67108863": Workload(
        "tanh3_f32_odd_67108863", "tanh", (3,), "f32", (67108863,), "uniform", 8.0, 1.0, 4,
        {"kind": "uniform", "A": -8.0, "B": 8.0, "n_grid": 3200}),
}

# The configuration the headline metric is quoted on: GELU 3-bit, bf16,
# [16, 2048, 8192].
HEADLINE = ("gelu_bf16_lm_ffn_16x2048x8192", 3)


def _storage_type(dtype: str):
    return np.uint32 if dtype == "f32" else np.uint16


def draw(dist: str, scale: float, n: int, dtype: str, seed: int, limit: int | None = None):
    """n (or the first `limit`) seeded draws as storage bit patterns.

    Works chunk by chunk in preallocated buffers (the values are those of
    one draw of the whole array)."""
    m = n if limit is None else min(n, limit)
    out = np.empty(m, _storage_type(dtype))
    rng = np.random.default_rng(seed)
    rng_mask = np.random.default_rng(seed + 2000) if dist == "mixture" else None
    cmax = min(CHUNK, max(m, 1))
    z = np.empty(cmax)
    u = np.empty(cmax) if dist == "mixture" else None
    f32 = np.empty(cmax, np.float32) if dtype == "bf16" else None
    pos = 0
    while pos < m:
        c = min(CHUNK, m - pos)
        zc = z[:c]
        if dist == "normal":
            rng.standard_normal(out=zc)
            zc *= scale
        elif dist == "mixture":
            rng.standard_normal(out=zc)
            zc *= scale
            rng_mask.random(out=u[:c])
            zc[u[:c] < 0.01] *= 10.0
        elif dist == "uniform":
            zc[...] = rng.uniform(-scale, scale, c)
        else:
            raise ValueError(dist)
        dst = out[pos:pos + c]
        if dtype == "f32":
            dst.view(np.float32)[...] = zc
        elif dtype == "f16":
            dst.view(np.float16)[...] = zc
        elif dtype == "bf16":
            import torch
            f32[:c] = zc
            torch.from_numpy(dst.view(np.int16)).view(torch.bfloat16).copy_(
                torch.from_numpy(f32[:c]))
        else:
            raise ValueError(dtype)
        pos += c
    return out


def inputs(w: Workload, limit: int | None = None):
    """(x_bits, g_bits) of workload w, as numpy storage arrays."""
    x = draw(w.x_dist, w.x_scale, w.n, w.dtype, w.seed, limit)
    g = draw("normal", w.g_sigma, w.n, w.dtype, w.seed + 1000, limit)
    return x, g
