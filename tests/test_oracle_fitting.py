"""Pins of the oracle's fitting net (descriptor -> energy) and its backward
dE/dD; each pin also rejects planted mistakes."""
import numpy as np

import oracle.fitting as fn
from synth.system import random_fitting_net


def _case(seed=0, n=3, M=6, m2=3, widths=(7, 7, 7)):
    rng = np.random.default_rng(seed)
    net = random_fitting_net(rng, M * m2, widths)
    D = rng.normal(size=(n, M, m2))
    return D, net


def _fd_error(bwd, D, net):
    g = bwd(D, net)
    h = 1e-6
    worst = 0.0
    for a in range(D.shape[0]):
        for m in range(D.shape[1]):
            for k in range(D.shape[2]):
                Dp = D.copy(); Dm = D.copy()
                Dp[a, m, k] += h; Dm[a, m, k] -= h
                fd = (fn.forward(Dp, net)[0][a] - fn.forward(Dm, net)[0][a]) / (2 * h)
                worst = max(worst, abs(fd - g[a, m, k]) / np.max(np.abs(g[a])))
    return worst


def _no_residual_grad(D, net):
    _, t = fn.forward(D, net)
    W = net["W"]
    delta = np.broadcast_to(net["w_out"], (D.shape[0], len(net["w_out"]))).copy()
    for l in (2, 1):
        delta = ((1.0 - t[l] ** 2) * delta) @ W[l].T          # dropped "delta +"
    return (((1.0 - t[0] ** 2) * delta) @ W[0].T).reshape(D.shape)


def _untransposed(D, net):
    _, t = fn.forward(D, net)
    W = net["W"]
    delta = np.broadcast_to(net["w_out"], (D.shape[0], len(net["w_out"]))).copy()
    for l in (2, 1):
        delta = delta + ((1.0 - t[l] ** 2) * delta) @ W[l]     # W instead of W^T
    return (((1.0 - t[0] ** 2) * delta) @ W[0].T).reshape(D.shape)


def test_backward_central_difference():
    D, net = _case()
    assert _fd_error(fn.backward, D, net) <= 1e-7
    for bad in (_no_residual_grad, _untransposed):
        assert _fd_error(bad, D, net) > 1e-3


def test_energy_is_per_atom():
    # E_i depends on D_i only: changing atom 1's descriptor leaves E_0 and E_2
    D, net = _case(1)
    E0, _ = fn.forward(D, net)
    D2 = D.copy(); D2[1] += 0.3
    E1, _ = fn.forward(D2, net)
    assert E1[0] == E0[0] and E1[2] == E0[2] and E1[1] != E0[1]


def test_single_hidden_layer_closed_form():
    # W_2 = W_3 = 0, b_2 = b_3 = 0: h_3 = h_1, E = tanh(x W_1 + b_1) . w + b,
    # dE/dx = W_1 ((1 - t^2) * w)
    D, net = _case(2)
    for l in (1, 2):
        net["W"][l][:] = 0.0
        net["b"][l][:] = 0.0
    x = D.reshape(len(D), -1)
    t = np.tanh(x @ net["W"][0] + net["b"][0])
    E, _ = fn.forward(D, net)
    np.testing.assert_allclose(E, t @ net["w_out"] + net["b_out"], rtol=1e-14)
    g = fn.backward(D, net).reshape(len(D), -1)
    np.testing.assert_allclose(g, ((1 - t ** 2) * net["w_out"]) @ net["W"][0].T, rtol=1e-13, atol=1e-15)


def test_residual_layers_closed_form():
    # W_2 = W_3 = 0 with nonzero biases: each residual layer adds the constant
    # tanh(b_l), so h_3 = h_1 + tanh(b_2) + tanh(b_3), and the gradient is that
    # of the first layer alone (the constant terms carry none)
    D, net = _case(3)
    for l in (1, 2):
        net["W"][l][:] = 0.0
    x = D.reshape(len(D), -1)
    t = np.tanh(x @ net["W"][0] + net["b"][0])
    h3 = t + np.tanh(net["b"][1]) + np.tanh(net["b"][2])
    E, _ = fn.forward(D, net)
    np.testing.assert_allclose(E, h3 @ net["w_out"] + net["b_out"], rtol=1e-14)
    g = fn.backward(D, net).reshape(len(D), -1)
    np.testing.assert_allclose(g, ((1 - t ** 2) * net["w_out"]) @ net["W"][0].T, rtol=1e-13, atol=1e-15)
    # a forward pass without the residual additions misses the first two terms
    h_plain = np.tanh(np.tanh(t @ net["W"][1] + net["b"][1]) @ net["W"][2] + net["b"][2])
    assert np.max(np.abs(h_plain @ net["w_out"] + net["b_out"] - E)) > 1e-2
