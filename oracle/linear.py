"""CPU oracle for the decode step's dense projections.

TEST INFRASTRUCTURE. Only the tests, the package smoke check and the bench's
CPU-baseline leg may import or call this module. The GPU library never does,
and this module imports nothing from the GPU path.

What it computes. Every decode step runs each layer's projections (QKV, O,
gate and up, down) and the LM head over the batch's current tokens; they
set the step's latency floor that the roofline batch bound B refers to
(§5.2) and the flat part of the latency-versus-batch figure (§2.4). The
operation is the plain product

    y[m, n] = sum_k x[m, k] * w[n, k]

with x [M, K] (one row per trajectory) and w [N, K] (one row per output
feature, the usual layout of a linear layer's weight), both bf16, in
float64 here.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits).astype(np.uint32) << np.uint32(16)).view(
        np.float32).astype(np.float64)


def linear(x_bits: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """y = x w^T in float64 from bf16 codes x [M, K], w [N, K]."""
    return bf16_to_f64(x_bits) @ bf16_to_f64(w_bits).T


def linear_abs(x_bits: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """sum_k |x[m, k] w[n, k]|: the scale of each output's rounding error."""
    return np.abs(bf16_to_f64(x_bits)) @ np.abs(bf16_to_f64(w_bits)).T
