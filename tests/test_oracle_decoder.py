"""Pins of the decode-step element-wise oracle (RMS norm, SwiGLU) against
closed forms, invariants, a plain-loop evaluation and scipy's logistic
function."""
import math

import numpy as np
import pytest
from scipy.special import expit

from oracle.decoder import rmsnorm, silu_mul
from oracle.linear import bf16_to_f64


def to_bits(a):
    """Exact bf16 codes of values that bf16 represents (checked)."""
    f = np.asarray(a, dtype=np.float32)
    bits = (f.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(bf16_to_f64(bits), f.astype(np.float64))
    return bits


def rand_bits(rng, shape):
    return (rng.standard_normal(shape).astype(np.float32).view(np.uint32)
            >> 16).astype(np.uint16)


def test_rmsnorm_plain_loops():
    rng = np.random.default_rng(0)
    x, w = rand_bits(rng, (3, 24)), rand_bits(rng, 24)
    xf, wf = bf16_to_f64(x), bf16_to_f64(w)
    got = rmsnorm(x, w, eps=1e-5)
    for m in range(3):
        ss = 0.0
        for k in range(24):
            ss += xf[m, k] * xf[m, k]
        r = 1.0 / math.sqrt(ss / 24 + 1e-5)
        for k in range(24):
            assert got[m, k] == pytest.approx(xf[m, k] * r * wf[k], rel=1e-14)


def test_rmsnorm_closed_forms_and_invariants():
    n = 64
    # a constant row is its sign times the weight (eps = 0)
    for c in (3.0, -0.5, 1024.0):
        y = rmsnorm(to_bits(np.full((1, n), c)), eps=0.0)
        assert np.allclose(y, np.sign(c), rtol=0, atol=1e-15)
    # a one-hot row: sqrt(n) at the hot index
    row = np.zeros((1, n)); row[0, 5] = -2.0
    y = rmsnorm(to_bits(row), eps=0.0)
    assert y[0, 5] == pytest.approx(-math.sqrt(n)) and np.count_nonzero(y) == 1
    # unit mean square without a weight; invariant under positive scaling
    rng = np.random.default_rng(1)
    x = rand_bits(rng, (4, n))
    y = rmsnorm(x, eps=0.0)
    assert np.allclose(np.mean(y * y, axis=1), 1.0, rtol=1e-14)
    x4 = to_bits(bf16_to_f64(x) * 4.0)                  # exact in bf16
    assert np.allclose(rmsnorm(x4, eps=0.0), y, rtol=1e-14)
    # the weight multiplies column-wise; eps shrinks toward zero
    w = rand_bits(rng, n)
    assert np.allclose(rmsnorm(x, w, eps=0.0), y * bf16_to_f64(w), rtol=1e-14)
    assert np.all(np.abs(rmsnorm(x, eps=1e6)) < np.abs(y))


def test_silu_mul_against_scipy_and_identities():
    rng = np.random.default_rng(2)
    gu = rand_bits(rng, (3, 2 * 40))
    g, u = bf16_to_f64(gu[:, :40]), bf16_to_f64(gu[:, 40:])
    got = silu_mul(gu)
    assert np.allclose(got, g * expit(g) * u, rtol=1e-14, atol=0)
    # silu(0) = 0; large gates pass through, very negative ones vanish
    gates = np.array([[0.0, 60.0, -60.0, 1.0]])
    y = silu_mul(to_bits(np.concatenate([gates, np.ones_like(gates)], axis=1)))
    assert y[0, 0] == 0.0 and y[0, 1] == pytest.approx(60.0)
    assert abs(y[0, 2]) < 1e-20
    assert y[0, 3] == pytest.approx(1.0 / (1.0 + math.exp(-1.0)))
    # silu(-g) = silu(g) - g
    gp = to_bits(np.concatenate([g, np.ones_like(g)], axis=1))
    gn = to_bits(np.concatenate([-g, np.ones_like(g)], axis=1))
    assert np.allclose(silu_mul(gn), silu_mul(gp) - g, rtol=1e-12, atol=1e-15)
