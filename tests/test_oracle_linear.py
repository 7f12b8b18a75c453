"""Pins of the projection oracle: brute-force triple loops on small shapes,
the identity weight, and linearity."""
import numpy as np
import torch

from oracle.linear import bf16_to_f64, linear, linear_abs


def bits(a):
    return torch.as_tensor(a, dtype=torch.float32).to(torch.bfloat16).view(
        torch.int16).numpy().view(np.uint16)


def test_brute_force_small():
    rng = np.random.default_rng(0)
    for m, n, k in ((1, 3, 5), (4, 7, 16), (3, 2, 1)):
        x, w = bits(rng.normal(size=(m, k))), bits(rng.normal(size=(n, k)))
        xf, wf = bf16_to_f64(x), bf16_to_f64(w)
        want = np.zeros((m, n))
        for i in range(m):
            for j in range(n):
                for t in range(k):
                    want[i, j] += xf[i, t] * wf[j, t]
        np.testing.assert_allclose(linear(x, w), want, rtol=1e-13, atol=1e-13)
        assert np.all(linear_abs(x, w) >= np.abs(want) - 1e-12)


def test_identity_weight_returns_x():
    rng = np.random.default_rng(1)
    x = bits(rng.normal(size=(5, 32)))
    np.testing.assert_array_equal(linear(x, bits(np.eye(32))), bf16_to_f64(x))


def test_linear_in_w():
    rng = np.random.default_rng(2)
    x = bits(rng.normal(size=(3, 64)))
    # values exactly representable in bf16 so that w1 + w2 is too
    w1 = bits(rng.integers(-8, 8, size=(9, 64)))
    w2 = bits(rng.integers(-8, 8, size=(9, 64)))
    w12 = bits(bf16_to_f64(w1) + bf16_to_f64(w2))
    np.testing.assert_allclose(linear(x, w12), linear(x, w1) + linear(x, w2),
                               rtol=1e-13, atol=1e-12)
