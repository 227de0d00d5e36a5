"""Pins of the oracle's descriptor backward dE/dT from dE/dD (paper Sec. II:
D_i = T_i (T_i<)^T).  Each pin is also run against planted mistakes (a
dropped term, a transposed index) to show that it would catch them."""
import numpy as np
import pytest

from oracle.se_a import backward, descriptor_backward, forward
from oracle.table import build_tables


def _D(T, m2):
    # D[m][n] = sum_k T[m][k] T[n][k], n < m2: the definition, for differencing
    return np.einsum("amk,ank->amn", T, T[:, :m2, :])


def _fd_error(fn, M=7, m2=3, seed=0):
    rng = np.random.default_rng(seed)
    T = rng.normal(size=(2, M, 4))
    W = rng.normal(size=(2, M, m2))
    dT = fn(T, W)
    h = 1e-6
    worst = 0.0
    for a in range(2):
        for m in range(M):
            for k in range(4):
                Tp = T.copy(); Tm = T.copy()
                Tp[a, m, k] += h; Tm[a, m, k] -= h
                fd = (np.sum(W * _D(Tp, m2)) - np.sum(W * _D(Tm, m2))) / (2 * h)
                worst = max(worst, abs(fd - dT[a, m, k]) / np.max(np.abs(dT[a])))
    return worst


# plausible mistakes, planted in copies
def _no_second_term(T, dD):
    return dD @ T[:, :dD.shape[2], :]


def _transposed(T, dD):
    m2 = dD.shape[2]
    dT = dD @ T[:, :m2, :]
    dT[:, :m2, :] += dD[:, :m2, :] @ T[:, :m2, :]      # dD[m][m'] instead of dD[m'][m]
    return dT


def test_central_difference():
    # E = <W, D(T)>: the backward against central differences of the definition
    assert _fd_error(descriptor_backward) <= 1e-8
    assert _fd_error(descriptor_backward, M=5, m2=5, seed=3) <= 1e-8
    assert _fd_error(descriptor_backward, M=6, m2=1, seed=4) <= 1e-8
    for bad in (_no_second_term, _transposed):
        assert _fd_error(bad) > 1e-3


def _unit_error(fn):
    # dE/dD = e_(p,q): D[p][q] = <T_p, T_q>, so dE/dT_p = T_q and dE/dT_q = T_p
    rng = np.random.default_rng(5)
    M, m2 = 6, 3
    T = rng.normal(size=(1, M, 4))
    worst = 0.0
    for p in range(M):
        for q in range(m2):
            dD = np.zeros((1, M, m2)); dD[0, p, q] = 1.0
            want = np.zeros((1, M, 4))
            want[0, p] += T[0, q]
            want[0, q] += T[0, p]
            worst = max(worst, np.max(np.abs(fn(T, dD) - want)))
    return worst


def test_unit_gradient_closed_form():
    assert _unit_error(descriptor_backward) <= 1e-15
    for bad in (_no_second_term, _transposed):
        assert _unit_error(bad) > 0.1


def test_symmetric_full_descriptor():
    # m2 = M and a symmetric dE/dD: dE/dT = 2 dE/dD T
    rng = np.random.default_rng(6)
    T = rng.normal(size=(3, 5, 4))
    S = rng.normal(size=(3, 5, 5)); S = S + np.transpose(S, (0, 2, 1))
    np.testing.assert_allclose(descriptor_backward(T, S), 2 * S @ T, rtol=0, atol=1e-13)


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_water"])
def test_chain_to_env_matrix(tiny_inputs, key):
    # E = <W, D(R~)>: dE/dR~ = backward(descriptor_backward(T, W)) vs central
    # differences of the oracle's forward D
    x = tiny_inputs[key]
    tabs = build_tables(x)
    rng = np.random.default_rng(8)
    atoms = np.arange(0, len(x.nlist), max(1, len(x.nlist) // 3))[:3]
    T, D = forward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2, atoms=atoms)
    W = rng.normal(size=D.shape)
    dT = np.zeros((len(x.nlist), x.cfg.m1, 4))
    dT[atoms] = descriptor_backward(T, W)
    dR = backward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, dT, atoms=atoms)
    h = 1e-6
    worst = 0.0
    for n, i in enumerate(atoms):
        js = np.nonzero(x.nlist[i] >= 0)[0]
        for j in js[rng.choice(len(js), size=min(4, len(js)), replace=False)]:
            for k in range(4):
                ep = x.em[i:i + 1].copy(); em_ = x.em[i:i + 1].copy()
                ep[0, j, k] += h; em_[0, j, k] -= h
                _, Dp = forward(ep, x.nlist[i:i + 1], x.atype[i:i + 1], tabs, x.cfg.sel, x.cfg.m2)
                _, Dm = forward(em_, x.nlist[i:i + 1], x.atype[i:i + 1], tabs, x.cfg.sel, x.cfg.m2)
                fd = (np.sum(W[n] * Dp[0]) - np.sum(W[n] * Dm[0])) / (2 * h)
                worst = max(worst, abs(fd - dR[n, j, k]) / np.max(np.abs(dR[n, j])))
    assert worst <= 1e-6, worst
