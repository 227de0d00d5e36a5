"""Pins of the oracle's forward (T, D) and backward (dE/dR~)."""
import numpy as np
import pytest

from oracle import cref
from oracle.se_a import backward, backward_untabulated, energy, forward, forward_untabulated
from oracle.table import build_tables


def _case(tiny_inputs, key):
    x = tiny_inputs[key]
    return x, build_tables(x)


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water"])
def test_forward_matches_untabulated_net(tiny_inputs, key):
    # fused tabulated T vs the original path with G materialised from the net
    x, tabs = _case(tiny_inputs, key)
    T, D, AT, AD = forward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2, with_abs=True)
    Tu, Du = forward_untabulated(x.em, x.nlist, x.atype, x.nets, x.cfg.sel, x.cfg.m2)
    assert np.all(np.abs(T - Tu) <= 1e-9 * AT + 1e-15)
    assert np.all(np.abs(D - Du) <= 1e-8 * AD + 1e-15)


def test_single_neighbour_closed_form(tiny_inputs):
    # one valid neighbour: T = g (x) r~ and D[m][n] = g_m g_n |r~|^2
    x, tabs = _case(tiny_inputs, "tiny_fcc")
    em = np.zeros_like(x.em[:1]); nl = np.full_like(x.nlist[:1], -1)
    r = np.array([0.37, -0.4, 0.25, 0.9])
    em[0, 5] = r; nl[0, 5] = 3
    T, D = forward(em, nl, x.atype[:1], tabs, x.cfg.sel, x.cfg.m2)
    g, _ = tabs[0].evaluate(np.array([r[0]]))
    np.testing.assert_allclose(T[0], np.outer(g[0], r), rtol=1e-15, atol=0)
    m2 = x.cfg.m2
    np.testing.assert_allclose(D[0], np.outer(g[0], g[0][:m2]) * (r @ r), rtol=1e-14, atol=1e-300)


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_water"])
def test_permutation_invariance(tiny_inputs, key):
    x, tabs = _case(tiny_inputs, key)
    rng = np.random.default_rng(0)
    em, nl = x.em.copy(), x.nlist.copy()
    off = np.concatenate([[0], np.cumsum(x.cfg.sel)])
    for i in range(len(nl)):
        for b in range(x.cfg.ntypes):
            p = off[b] + rng.permutation(x.cfg.sel[b])
            em[i, off[b]:off[b + 1]] = x.em[i, p]
            nl[i, off[b]:off[b + 1]] = x.nlist[i, p]
    T0, D0 = forward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    T1, D1 = forward(em, nl, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    scale = np.max(np.abs(T0), axis=(1, 2), keepdims=True)
    assert np.max(np.abs(T1 - T0) / scale) < 1e-14


def test_padding_rows_contribute_nothing(tiny_inputs):
    # move the valid rows of each block to the end of the block (same order):
    # T is bit-identical; and garbage in padded rows is ignored entirely
    x, tabs = _case(tiny_inputs, "tiny_alloy")
    em = np.zeros_like(x.em); nl = np.full_like(x.nlist, -1)
    off = np.concatenate([[0], np.cumsum(x.cfg.sel)])
    for i in range(len(nl)):
        for b in range(x.cfg.ntypes):
            v = off[b] + np.nonzero(x.nlist[i, off[b]:off[b + 1]] >= 0)[0]
            dst = np.arange(off[b + 1] - len(v), off[b + 1])
            em[i, dst] = x.em[i, v]; nl[i, dst] = x.nlist[i, v]
    T0, D0 = forward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    T1, D1 = forward(em, nl, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    np.testing.assert_array_equal(T0, T1)
    em2 = x.em.copy(); em2[x.nlist < 0] = 123.0
    T2, _ = forward(em2, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    np.testing.assert_array_equal(T0, T2)


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy"])
def test_rotation_covariance(tiny_inputs, key):
    # rotating the spatial columns of R~ rotates T[:, :, 1:] and leaves D invariant
    x, tabs = _case(tiny_inputs, key)
    q, _ = np.linalg.qr(np.random.default_rng(5).normal(size=(3, 3)))
    em = x.em.copy(); em[..., 1:] = x.em[..., 1:] @ q.T
    T0, D0 = forward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    T1, D1 = forward(em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    sT = np.max(np.abs(T0)); sD = np.max(np.abs(D0))
    np.testing.assert_allclose(T1[..., 0], T0[..., 0], rtol=0, atol=1e-14 * sT)
    np.testing.assert_allclose(T1[..., 1:], T0[..., 1:] @ q.T, rtol=0, atol=1e-13 * sT)
    np.testing.assert_allclose(D1, D0, rtol=0, atol=1e-12 * sD)


def test_linear_in_spatial_columns(tiny_inputs):
    x, tabs = _case(tiny_inputs, "tiny_water")
    em = x.em.copy(); em[..., 1:] *= 2.5
    T0, _ = forward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    T1, _ = forward(em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    np.testing.assert_array_equal(T1[..., 0], T0[..., 0])
    np.testing.assert_allclose(T1[..., 1:], 2.5 * T0[..., 1:], rtol=1e-14, atol=1e-14)


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_water", "tiny_alloy"])
def test_backward_central_difference(tiny_inputs, key):
    # E = <Lambda, T(R~)>; dE/dR~ from the backward vs central differences
    x, tabs = _case(tiny_inputs, key)
    atoms = np.arange(0, len(x.nlist), max(1, len(x.nlist) // 6))[:6]
    rng = np.random.default_rng(9)
    lam = rng.normal(size=(len(x.nlist), x.cfg.m1, 4))
    dR = backward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, lam, atoms=atoms)
    h = 1e-6
    worst = 0.0
    for n, i in enumerate(atoms):
        js = np.nonzero(x.nlist[i] >= 0)[0]
        for j in js[rng.choice(len(js), size=min(6, len(js)), replace=False)]:
            for k in range(4):
                ep = x.em[i:i + 1].copy(); em_ = x.em[i:i + 1].copy()
                ep[0, j, k] += h; em_[0, j, k] -= h
                Tp, _ = forward(ep, x.nlist[i:i + 1], x.atype[i:i + 1], tabs, x.cfg.sel, x.cfg.m2)
                Tm, _ = forward(em_, x.nlist[i:i + 1], x.atype[i:i + 1], tabs, x.cfg.sel, x.cfg.m2)
                fd = (energy(Tp, lam[i:i + 1]) - energy(Tm, lam[i:i + 1])) / (2 * h)
                scale = np.max(np.abs(dR[n, j]))
                worst = max(worst, abs(fd - dR[n, j, k]) / scale)
    assert worst <= 1e-6, worst


def test_backward_padding_rows_zero(tiny_inputs):
    x, tabs = _case(tiny_inputs, "tiny_alloy")
    lam = np.random.default_rng(1).normal(size=(len(x.nlist), x.cfg.m1, 4))
    dR = backward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, lam)
    assert np.all(dR[x.nlist < 0] == 0)


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water"])
def test_c_oracle_matches_numpy_oracle(tiny_inputs, key):
    x, tabs = _case(tiny_inputs, key)
    pb = cref.Problem(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    T, D = pb.forward()
    T0, D0 = forward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    np.testing.assert_allclose(T, T0, rtol=0, atol=1e-13 * np.max(np.abs(T0)))
    np.testing.assert_allclose(D, D0, rtol=0, atol=1e-13 * np.max(np.abs(D0)))
    lam = np.random.default_rng(2).normal(size=(len(x.nlist), x.cfg.m1, 4))
    dR = pb.backward(lam)
    dR0 = backward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, lam)
    np.testing.assert_allclose(dR, dR0, rtol=0, atol=1e-13 * np.max(np.abs(dR0)))
    # chunked ranges give the same rows
    T2, _ = pb.forward(7, 19)
    np.testing.assert_array_equal(T2, T[7:19])


def test_backward_untabulated_central_difference(tiny_inputs):
    # E = <Lambda, T(R~)> through the real net: against central differences of
    # forward_untabulated, and close to the tabulated backward
    x, tabs = _case(tiny_inputs, "tiny_water")
    atoms = np.arange(0, len(x.nlist), max(1, len(x.nlist) // 4))[:4]
    rng = np.random.default_rng(12)
    lam = rng.normal(size=(len(x.nlist), x.cfg.m1, 4))
    dR = backward_untabulated(x.em, x.nlist, x.atype, x.nets, x.cfg.sel, lam, atoms=atoms)
    dRt = backward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, lam, atoms=atoms)
    assert np.max(np.abs(dR - dRt)) <= 1e-8 * np.max(np.abs(dR))
    h = 1e-6
    worst = 0.0
    for n, i in enumerate(atoms):
        js = np.nonzero(x.nlist[i] >= 0)[0]
        for j in js[rng.choice(len(js), size=min(4, len(js)), replace=False)]:
            for k in range(4):
                ep = x.em[i:i + 1].copy(); em_ = x.em[i:i + 1].copy()
                ep[0, j, k] += h; em_[0, j, k] -= h
                Tp, _ = forward_untabulated(ep, x.nlist[i:i + 1], x.atype[i:i + 1], x.nets, x.cfg.sel, x.cfg.m2)
                Tm, _ = forward_untabulated(em_, x.nlist[i:i + 1], x.atype[i:i + 1], x.nets, x.cfg.sel, x.cfg.m2)
                fd = (energy(Tp, lam[i:i + 1]) - energy(Tm, lam[i:i + 1])) / (2 * h)
                worst = max(worst, abs(fd - dR[n, j, k]) / np.max(np.abs(dR[n, j])))
    assert worst <= 1e-6, worst
