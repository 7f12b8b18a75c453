"""Pins of the roofline batch-bound oracle: a linear scan with exact
fractions, the closed form without activation traffic
(ceil(wb F / (2 BW)), 313 on MI355X bf16), the published non-embedding
parameter count of Qwen2.5-7B, and the shape of the step-time curve."""
from fractions import Fraction

import pytest

from oracle.roofline import (QWEN25_7B, QWEN25_32B, ModelShape, batch_bound,
                             params, projections, projections_compute_bound,
                             step_time)

MI355X_BF16_FLOPS = 2_500_000_000_000_000      # dense bf16 matrix cores
MI355X_HBM = 8_000_000_000_000                  # bytes per second


def scan(m, f, bw, limit=100_000):
    for batch in range(1, limit):
        if projections_compute_bound(m, batch, f, bw):
            return batch
    return None


@pytest.mark.parametrize("m", [QWEN25_7B, QWEN25_32B,
                               ModelShape(2, 64, 4, 2, 16, 128, 100),
                               ModelShape(3, 96, 6, 1, 32, 300, 50, 1, 1, 1)])
@pytest.mark.parametrize("f,bw", [(MI355X_BF16_FLOPS, MI355X_HBM),
                                  (5_000_000_000_000_000, MI355X_HBM),
                                  (10 ** 12, 10 ** 12)])
def test_bound_equals_a_linear_scan(m, f, bw):
    assert batch_bound(m, f, bw) == scan(m, f, bw)


def test_closed_form_without_activation_traffic():
    """ab = 0: the projections turn compute-bound at ceil(wb F / (2 BW))
    for any shape."""
    for m in (QWEN25_7B, QWEN25_32B, ModelShape(1, 8, 1, 1, 8, 8, 8)):
        m0 = ModelShape(**{**m.__dict__, "act_bytes": 0})
        assert batch_bound(m0, MI355X_BF16_FLOPS, MI355X_HBM) == 313
        assert batch_bound(m0, 4 * 10 ** 12, 10 ** 12) == 4
        m1 = ModelShape(**{**m0.__dict__, "weight_bytes": 1})   # fp8 weights
        assert batch_bound(m1, 5_000_000_000_000_000, MI355X_HBM) == 313


def test_qwen7b_parameter_count():
    # published non-embedding parameters of Qwen2.5-7B: 6.53B, plus the
    # untied LM head (3584 x 152064)
    assert round((params(QWEN25_7B) - 3584 * 152064) / 1e9, 2) == 6.53
    assert len(projections(QWEN25_7B)) == 4 * 28 + 1


def test_activations_push_the_bound_up_and_can_remove_it():
    m = QWEN25_7B
    with_act = batch_bound(m, MI355X_BF16_FLOPS, MI355X_HBM)
    m0 = ModelShape(**{**m.__dict__, "act_bytes": 0})
    assert with_act > batch_bound(m0, MI355X_BF16_FLOPS, MI355X_HBM)
    # tiny matrices with fat activations never become compute-bound
    tiny = ModelShape(1, 2, 1, 1, 2, 2, 2, 2, 64, 2)
    assert batch_bound(tiny, 10 ** 12, 10 ** 12) is None


def test_step_time_is_nearly_flat_below_the_bound():
    """Without context the step is the projections alone: nearly flat up to
    B, then growing with the batch (compute-bound). With context the KV
    reads add a cost per trajectory at every batch size."""
    f, bw = MI355X_BF16_FLOPS, MI355X_HBM
    b = batch_bound(QWEN25_7B, f, bw)
    t1 = step_time(QWEN25_7B, 1, 0, f, bw)
    assert step_time(QWEN25_7B, b, 0, f, bw) / t1 < Fraction(12, 10)
    assert step_time(QWEN25_7B, 4 * b, 0, f, bw) / t1 > Fraction(3)
    kv = Fraction(2 * 2 * 4 * 128 * 28 * 2048, bw)   # 2048 more cached tokens
    for m in (1, 64, b):
        assert (step_time(QWEN25_7B, m, 2048, f, bw)
                - step_time(QWEN25_7B, m, 0, f, bw)) == m * kv
