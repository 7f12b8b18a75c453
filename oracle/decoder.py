"""CPU oracle for the element-wise operations of a decode step.

TEST INFRASTRUCTURE. Only the tests, the package smoke check and the bench's
CPU-baseline leg may import or call this module. The GPU library never does,
and this module imports nothing from the GPU path.

What it computes. The decode-latency curve (§2.4) and the roofline batch
bound B of Algorithm 1 (§5.2) concern whole decode steps of the paper's
rollout models (Qwen2.5, §8 "Models"). Besides the projections and the
attention, each layer of those models runs an RMS pre-norm before its
attention and its MLP, and a gated (SwiGLU) activation inside the MLP. The
paper does not restate these definitions; they are the models' own:

    rmsnorm(x)[k]  = x[k] / sqrt(mean_j x[j]^2 + eps) * w[k]
    silu_mul(g, u) = g / (1 + exp(-g)) * u

computed here in float64 from the bf16 codes of the inputs.
"""
from __future__ import annotations

import numpy as np

from .linear import bf16_to_f64


def rmsnorm(x_bits: np.ndarray, w_bits=None, eps: float = 1e-6) -> np.ndarray:
    """Row-wise RMS norm of x [M, N] (bf16 codes), times w [N] if given."""
    x = bf16_to_f64(x_bits)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    y = x * r
    if w_bits is not None:
        y = y * bf16_to_f64(w_bits)
    return y


def silu_mul(gu_bits: np.ndarray) -> np.ndarray:
    """gu [M, 2I] (bf16 codes, gate then up) -> silu(gate) * up [M, I]."""
    gu = bf16_to_f64(gu_bits)
    i = gu.shape[-1] // 2
    g, u = gu[..., :i], gu[..., i:]
    return g / (1.0 + np.exp(-g)) * u
