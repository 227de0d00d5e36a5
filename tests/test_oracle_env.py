"""Pins of the oracle's environment matrix and force / virial assembly
(paper Sec. II, Eq. (1) and the normalisation after it; F = -dE/dr)."""
import numpy as np
import pytest

import oracle.env as ev


def _stats(x):
    s = x.stats
    return s["mean"], s["sigma"], s["sigma_all"]


def test_weight_closed_forms_and_smoothness():
    rc, rcs = 6.0, 0.5
    r = np.array([0.2, 0.49, 1.0, 3.0, 5.99, 6.0, 7.0])
    s, ds = ev.weight(r, rc, rcs)
    np.testing.assert_allclose(s[:2], 1.0 / r[:2], rtol=1e-15)
    np.testing.assert_allclose(ds[:2], -1.0 / r[:2] ** 2, rtol=1e-15)
    assert s[5] == 0.0 and s[6] == 0.0 and ds[6] == 0.0
    # C^1 at r_cs and r_c: values and slopes meet from both sides
    for x0 in (rcs, rc):
        e = 1e-7
        sl, dl = ev.weight(np.array([x0 - e]), rc, rcs)
        sr, dr = ev.weight(np.array([x0 + e]), rc, rcs)
        assert abs(sl[0] - sr[0]) < 1e-5 and abs(dl[0] - dr[0]) < 1e-4
    # ds/dr against central differences inside each piece
    for x0 in (0.3, 1.7, 4.2, 5.9):
        h = 1e-6
        fd = (ev.weight(np.array([x0 + h]), rc, rcs)[0][0] - ev.weight(np.array([x0 - h]), rc, rcs)[0][0]) / (2 * h)
        assert abs(fd - ev.weight(np.array([x0]), rc, rcs)[1][0]) < 1e-7


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_water", "tiny_alloy"])
def test_env_mat_matches_generator(tiny_inputs, key):
    # the generator builds R~ from its own displacement vectors; the oracle
    # from positions by minimum image
    x = tiny_inputs[key]
    em = ev.env_mat(x.coords, x.cfg.box, x.atype, x.nlist, x.cfg.rc, x.cfg.rcs, *_stats(x))
    assert np.max(np.abs(em - x.em)) <= 1e-12 * np.max(np.abs(x.em))
    assert np.all(em[x.nlist < 0] == 0)


def _case(tiny_inputs, key="tiny_water", seed=3):
    x = tiny_inputs[key]
    lam = np.random.default_rng(seed).normal(size=x.em.shape) * (x.nlist >= 0)[..., None]
    return x, lam


def _energy(x, lam, coords):
    em = ev.env_mat(coords, x.cfg.box, x.atype, x.nlist, x.cfg.rc, x.cfg.rcs, *_stats(x))
    return float(np.sum(lam * em))


def _force_fd_error(x, lam, force_fn):
    F, _ = force_fn(x.coords, x.cfg.box, x.atype, x.nlist, x.cfg.rc, x.cfg.rcs, *_stats(x), lam)
    h = 1e-6
    worst = 0.0
    for i in (0, 7, len(x.coords) - 1):
        for a in range(3):
            cp = x.coords.copy(); cm = x.coords.copy()
            cp[i, a] += h; cm[i, a] -= h
            fd = -(_energy(x, lam, cp) - _energy(x, lam, cm)) / (2 * h)
            worst = max(worst, abs(fd - F[i, a]) / np.max(np.abs(F[i])))
    return worst


def _wrong_sign_scatter(coords, box, atype, nlist, rc, rcs, mean, sigma, sigma_all, lam):
    F, V = ev.force_virial(coords, box, atype, nlist, rc, rcs, mean, sigma, sigma_all, lam)
    valid = nlist >= 0
    g = ev.pair_gradients(ev.pair_vectors(coords, box, nlist), valid, atype, rc, rcs, sigma, sigma_all, lam)
    for i in range(len(nlist)):
        for s in np.nonzero(valid[i])[0]:
            F[nlist[i, s]] += 2 * g[i, s]               # F_j += g instead of -= g
    return F, V


def _no_delta_term(coords, box, atype, nlist, rc, rcs, mean, sigma, sigma_all, lam):
    lam2 = lam.copy(); lam2[..., 1:] = 0.0             # drops d(s x)/dr entirely
    return ev.force_virial(coords, box, atype, nlist, rc, rcs, mean, sigma, sigma_all, lam2)


def test_forces_central_difference(tiny_inputs):
    x, lam = _case(tiny_inputs)
    assert _force_fd_error(x, lam, ev.force_virial) <= 1e-6
    for bad in (_wrong_sign_scatter, _no_delta_term):
        assert _force_fd_error(x, lam, bad) > 1e-2


def test_forces_sum_to_zero(tiny_inputs):
    # E depends on differences of positions only
    x, lam = _case(tiny_inputs, "tiny_alloy", 4)
    F, _ = ev.force_virial(x.coords, x.cfg.box, x.atype, x.nlist, x.cfg.rc, x.cfg.rcs, *_stats(x), lam)
    assert np.max(np.abs(F.sum(0))) <= 1e-11 * np.max(np.abs(F))


def test_virial_central_difference_of_strain(tiny_inputs):
    # sum_i V_i[a][b] = -dE/d eps_ba for r_ij -> (1 + eps) r_ij
    x, lam = _case(tiny_inputs, "tiny_fcc", 5)
    mean, sigma, sigma_all = _stats(x)
    _, V = ev.force_virial(x.coords, x.cfg.box, x.atype, x.nlist, x.cfg.rc, x.cfg.rcs, mean, sigma, sigma_all, lam)
    W = V.sum(0)
    rij = ev.pair_vectors(x.coords, x.cfg.box, x.nlist)
    valid = x.nlist >= 0

    def energy(eps):
        r2 = rij @ (np.eye(3) + eps).T
        em = ev.rows_from_vectors(r2, valid, x.atype, x.cfg.rc, x.cfg.rcs, mean, sigma, sigma_all)
        return float(np.sum(lam * em))
    h = 1e-6
    for b in range(3):
        for a in range(3):
            e = np.zeros((3, 3)); e[b, a] = h
            fd = (energy(e) - energy(-e)) / (2 * h)
            assert abs(-fd - W[a, b]) <= 1e-6 * np.max(np.abs(W))


def test_env_mat_of_selected_atoms(tiny_inputs):
    # rows of a subset of atoms equal the same rows of the whole system
    x = tiny_inputs["tiny_alloy"]
    c = x.cfg
    full = ev.env_mat(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, *_stats(x))
    atoms = np.array([3, 0, 11])
    part = ev.env_mat(x.coords, c.box, x.atype[atoms], x.nlist[atoms], c.rc, c.rcs, *_stats(x), atoms=atoms)
    assert np.array_equal(part, full[atoms])


def test_chain_positions_to_forces(tiny_inputs):
    # E = <W, D(T(R~(r)))>: forces from the oracle's chain (descriptor
    # backward, backward, force assembly) against central differences of E
    # in the positions
    from oracle.se_a import backward, descriptor_backward, forward
    from oracle.table import build_tables
    x = tiny_inputs["tiny_water"]
    c = x.cfg
    tabs = build_tables(x)
    mean, sigma, sigma_all = _stats(x)

    def energy(coords, W):
        em = ev.env_mat(coords, c.box, x.atype, x.nlist, c.rc, c.rcs, mean, sigma, sigma_all)
        _, D = forward(em, x.nlist, x.atype, tabs, c.sel, c.m2)
        return float(np.sum(W * D)), em
    W = np.random.default_rng(7).normal(size=(len(x.atype), c.m1, c.m2))
    _, em = energy(x.coords, W)
    T, _ = forward(em, x.nlist, x.atype, tabs, c.sel, c.m2)
    dR = backward(em, x.nlist, x.atype, tabs, c.sel, descriptor_backward(T, W))
    F, _ = ev.force_virial(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, mean, sigma, sigma_all, dR)
    h = 1e-6
    for i in (0, 5):
        for a in range(3):
            cp = x.coords.copy(); cm = x.coords.copy()
            cp[i, a] += h; cm[i, a] -= h
            fd = -(energy(cp, W)[0] - energy(cm, W)[0]) / (2 * h)
            assert abs(fd - F[i, a]) <= 1e-5 * np.max(np.abs(F[i])), (i, a, fd, F[i, a])


def test_chain_with_fitting_net(tiny_inputs):
    # E = sum_i E_i(D_i(r)) through the fitting net: forces from the oracle's
    # chain against central differences of E in the positions
    import oracle.fitting as fn
    from oracle.se_a import backward, descriptor_backward, forward
    from oracle.table import build_tables
    from synth.system import random_fitting_net
    x = tiny_inputs["tiny_water"]
    c = x.cfg
    tabs = build_tables(x)
    mean, sigma, sigma_all = _stats(x)
    net = random_fitting_net(np.random.default_rng(8), c.m1 * c.m2, (12, 12, 12))

    def energy(coords):
        em = ev.env_mat(coords, c.box, x.atype, x.nlist, c.rc, c.rcs, mean, sigma, sigma_all)
        T, D = forward(em, x.nlist, x.atype, tabs, c.sel, c.m2)
        return float(np.sum(fn.forward(D, net)[0])), em, T, D
    _, em, T, D = energy(x.coords)
    dR = backward(em, x.nlist, x.atype, tabs, c.sel, descriptor_backward(T, fn.backward(D, net)))
    F, _ = ev.force_virial(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, mean, sigma, sigma_all, dR)
    h = 1e-6
    for i in (1, 6):
        for a in range(3):
            cp = x.coords.copy(); cm = x.coords.copy()
            cp[i, a] += h; cm[i, a] -= h
            fd = -(energy(cp)[0] - energy(cm)[0]) / (2 * h)
            assert abs(fd - F[i, a]) <= 1e-5 * np.max(np.abs(F[i])), (i, a, fd, F[i, a])
