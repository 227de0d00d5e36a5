"""The pins are sensitive: plausible mistakes planted in (copies of) the
oracle's arithmetic make them fail.  Everything here runs on the CPU."""
import numpy as np
import pytest

import oracle.table as ot
from oracle.net import embed, embed_d2
from oracle.se_a import backward, forward, energy
from synth.system import random_net

_HERMITE = ot.hermite_coefficients


def _reproduction_error(coef_fn):
    rng = np.random.default_rng(7)
    polys = [np.poly1d(c) for c in rng.normal(size=(3, 6))]
    func = lambda x: (np.stack([p(x) for p in polys], 1),
                      np.stack([p.deriv(1)(x) for p in polys], 1),
                      np.stack([p.deriv(2)(x) for p in polys], 1))
    orig = ot.hermite_coefficients
    ot.hermite_coefficients = coef_fn
    try:
        tab = ot.build_table_from(func, -0.7, 0.05, 40, 0.2, 8)
    finally:
        ot.hermite_coefficients = orig
    x = np.linspace(-0.7, tab.x_up, 501)
    return max(np.max(np.abs(tab.evaluate(x)[0][:, m] - p(x))) for m, p in enumerate(polys))


def test_reproduction_pin_catches_coefficient_mistakes():
    assert _reproduction_error(_HERMITE) < 1e-10

    def wrong_b(y0, dy0, d2y0, y1, dy1, d2y1, dt):      # 16 -> 15 in b
        a, b, c, d, e, f = _HERMITE(y0, dy0, d2y0, y1, dy1, d2y1, dt)
        return a, b - dy0 * dt / (2 * dt ** 4), c, d, e, f

    def wrong_c_sign(y0, dy0, d2y0, y1, dy1, d2y1, dt):  # + instead of - on the y'' term
        a, b, c, d, e, f = _HERMITE(y0, dy0, d2y0, y1, dy1, d2y1, dt)
        return a, b, c + (3 * d2y0 - d2y1) * dt ** 2 / dt ** 3, d, e, f

    def x_not_offset(y0, dy0, d2y0, y1, dy1, d2y1, dt):  # d = y'' instead of y''/2
        a, b, c, d, e, f = _HERMITE(y0, dy0, d2y0, y1, dy1, d2y1, dt)
        return a, b, c, 2 * d, e, f

    for bad in (wrong_b, wrong_c_sign, x_not_offset):
        assert _reproduction_error(bad) > 1e-6


def test_tabulation_pin_catches_off_by_one_interval():
    net = random_net(np.random.default_rng(0), (1, 25, 50, 100))
    tab = ot.build_table(net, -0.8, 0.01, 400, 0.1, 40)
    x = np.random.default_rng(1).uniform(-0.8, tab.x_up, 2000)
    assert np.max(np.abs(tab.evaluate(x)[0] - embed(x, net))) < 1e-9
    orig = ot.Table.locate

    def shifted(self, xx):
        l, t, c = orig(self, xx)
        l2 = np.minimum(l + 1, self.L1 + self.L2 - 1)
        return l2, t, c
    ot.Table.locate = shifted
    try:
        err = np.max(np.abs(tab.evaluate(x)[0] - embed(x, net)))
    finally:
        ot.Table.locate = orig
    assert err > 1e-6


def test_fd_pin_catches_missing_derivative_term(tiny_inputs):
    x = tiny_inputs["tiny_fcc"]
    tabs = ot.build_tables(x)
    i = 3
    lam = np.random.default_rng(2).normal(size=(len(x.nlist), x.cfg.m1, 4))
    j = int(np.nonzero(x.nlist[i] >= 0)[0][4])
    h = 1e-6
    ep = x.em[i:i + 1].copy(); em_ = x.em[i:i + 1].copy()
    ep[0, j, 0] += h; em_[0, j, 0] -= h
    fd = (energy(forward(ep, x.nlist[i:i + 1], x.atype[i:i + 1], tabs, x.cfg.sel, 4)[0], lam[i:i + 1])
          - energy(forward(em_, x.nlist[i:i + 1], x.atype[i:i + 1], tabs, x.cfg.sel, 4)[0], lam[i:i + 1])) / (2 * h)
    good = backward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, lam, atoms=[i])[0, j, 0]
    assert abs(fd - good) <= 1e-6 * abs(good)
    # dropping the g' term (x enters through g) is a large error
    g, gp = tabs[0].evaluate(np.array([x.em[i, j, 0]]))
    assert abs(fd - (good - gp[0] @ (lam[i] @ x.em[i, j]))) > 1e-3 * abs(good)


def test_closed_form_pin_catches_wrong_rows_of_D(tiny_inputs):
    x = tiny_inputs["tiny_fcc"]
    tabs = ot.build_tables(x)
    em = np.zeros_like(x.em[:1]); nl = np.full_like(x.nlist[:1], -1)
    r = np.array([0.37, -0.4, 0.25, 0.9]); em[0, 5] = r; nl[0, 5] = 3
    T, D = forward(em, nl, x.atype[:1], tabs, x.cfg.sel, x.cfg.m2)
    g = tabs[0].evaluate(np.array([r[0]]))[0][0]
    M2 = x.cfg.m2
    last_rows = np.outer(g, g[-M2:]) * (r @ r)       # D from the last M' rows
    assert np.max(np.abs(D[0] - last_rows)) > 1e-3 * np.max(np.abs(D[0]))
