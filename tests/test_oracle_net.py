"""Pins of the oracle's embedding net and its forward-mode derivatives."""
import numpy as np
import pytest

from oracle.net import embed, embed_d2
from synth.system import random_net


def _net(seed, widths=(1, 25, 50, 100)):
    return random_net(np.random.default_rng(seed), widths)


def test_single_layer_closed_form():
    # G = tanh(w x + b): G' = w (1 - G^2), G'' = -2 w^2 G (1 - G^2)
    rng = np.random.default_rng(1)
    w = rng.normal(size=(1, 7)); b = rng.normal(size=7)
    net = {"W": [w], "b": [b]}
    x = np.linspace(-3, 3, 41)
    y, dy, d2y = embed_d2(x, net)
    G = np.tanh(x[:, None] * w[0] + b)
    np.testing.assert_allclose(y, G, rtol=0, atol=1e-15)
    np.testing.assert_allclose(dy, w[0] * (1 - G * G), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(d2y, -2 * w[0] ** 2 * G * (1 - G * G), rtol=1e-13, atol=1e-14)


def test_residual_doubling_closed_form():
    # widths 1->2->4 with W = 0: each doubling layer adds [y, y] + tanh(b),
    # so G(x) = x + tanh(b1)[m % 2] + tanh(b2)[m] exactly, G' = 1, G'' = 0.
    b1 = np.array([0.3, -0.7]); b2 = np.array([0.1, 0.2, -0.4, 0.9])
    net = {"W": [np.zeros((1, 2)), np.zeros((2, 4))], "b": [b1, b2]}
    x = np.array([-1.5, 0.0, 0.25, 2.0])
    y, dy, d2y = embed_d2(x, net)
    expect = x[:, None] + np.tanh(b1)[[0, 1, 0, 1]] + np.tanh(b2)
    np.testing.assert_allclose(y, expect, rtol=0, atol=1e-15)
    np.testing.assert_array_equal(dy, np.ones_like(dy))
    np.testing.assert_array_equal(d2y, np.zeros_like(d2y))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_derivatives_complex_step(seed):
    # complex step: f'(x) = Im f(x + i h) / h exactly up to rounding (f analytic)
    net = _net(seed)
    x = np.linspace(-1.5, 6.5, 57)
    h = 1e-30
    y, dy, d2y = embed_d2(x, net)
    yc, dyc, _ = embed_d2(x + 1j * h, net)
    np.testing.assert_allclose(np.real(yc), y, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(np.imag(yc) / h, dy, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(np.imag(dyc) / h, d2y, rtol=1e-11, atol=1e-12)


def test_derivatives_central_difference():
    net = _net(5)
    x = np.linspace(-1, 5, 13)
    eps = 1e-5
    _, dy, d2y = embed_d2(x, net)
    fd1 = (embed(x + eps, net) - embed(x - eps, net)) / (2 * eps)
    fd2 = (embed(x + eps, net) - 2 * embed(x, net) + embed(x - eps, net)) / eps ** 2
    np.testing.assert_allclose(fd1, dy, rtol=1e-7, atol=1e-8)
    np.testing.assert_allclose(fd2, d2y, rtol=1e-3, atol=1e-4)


def test_embed_matches_embed_d2_value():
    net = _net(3)
    x = np.linspace(-2, 4, 9)
    np.testing.assert_array_equal(embed(x, net), embed_d2(x, net)[0])
