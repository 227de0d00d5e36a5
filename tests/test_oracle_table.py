"""Pins of the oracle's Hermite table (paper Sec. II closed forms)."""
import json
import math
import os

import numpy as np
import pytest

from oracle.net import embed, embed_d2
from oracle.table import build_table, build_table_from, hermite_coefficients
from synth.system import random_net

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _poly_func(coeffs):
    """Exact y, y', y'' of polynomials with rows of coefficients (highest
    power first), as an [n, M] vector function."""
    polys = [np.poly1d(c) for c in coeffs]

    def f(x):
        return (np.stack([p(x) for p in polys], 1),
                np.stack([p.deriv(1)(x) for p in polys], 1),
                np.stack([p.deriv(2)(x) for p in polys], 1))
    return f, polys


def test_golden_x5():
    # hand-derived Taylor coefficients of x^5 (tests/golden/quintic_x5.json)
    cases = json.load(open(os.path.join(GOLDEN, "quintic_x5.json")))["cases"]
    for c in cases:
        x0, dt = c["x_l"], c["dt"]
        x1 = x0 + dt
        got = hermite_coefficients(x0 ** 5, 5 * x0 ** 4, 20 * x0 ** 3,
                                   x1 ** 5, 5 * x1 ** 4, 20 * x1 ** 3, dt)
        np.testing.assert_allclose(got, c["abcdef"], rtol=1e-12, atol=1e-12)


def test_quintic_reproduced_exactly():
    # any polynomial of degree <= 5 is reproduced; its coefficients are the
    # Taylor coefficients at the left node: f=p, e=p', d=p''/2, ..., a=p5/120
    rng = np.random.default_rng(7)
    coeffs = rng.normal(size=(6, 6))
    coeffs[3, :2] = 0.0   # one cubic, one quartic, ...
    coeffs[4, :1] = 0.0
    func, polys = _poly_func(coeffs)
    tab = build_table_from(func, lo=-0.7, d1=0.05, L1=40, d2=0.2, L2=8)
    x = np.concatenate([np.linspace(-0.7, tab.x_end - 1e-9, 2001), [-0.7, tab.x_up]])
    g, g1, g2 = tab.evaluate(x, order=2)
    for m, p in enumerate(polys):
        scale = np.max(np.abs(p(x))) + 1
        np.testing.assert_allclose(g[:, m], p(x), rtol=0, atol=1e-11 * scale)
        np.testing.assert_allclose(g1[:, m], p.deriv(1)(x), rtol=0, atol=1e-9 * scale)
        np.testing.assert_allclose(g2[:, m], p.deriv(2)(x), rtol=0, atol=1e-7 * scale)
    # coefficients vs Taylor coefficients at a few nodes
    for l in (0, 17, 39, 40, 47):
        xl = (-0.7 + l * 0.05) if l < 40 else (tab.x_up + (l - 40) * 0.2)
        for m, p in enumerate(polys):
            taylor = [p.deriv(q)(xl) / math.factorial(q) if q else p(xl) for q in range(6)]
            np.testing.assert_allclose(tab.coef[l, m], taylor, rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("seed", [0, 1])
def test_c2_continuity_at_nodes(seed):
    # the quintic of interval l takes (y, y', y'') of node l+1 at t = dt
    net = random_net(np.random.default_rng(seed), (1, 25, 50, 100))
    tab = build_table(net, lo=-0.6, d1=0.01, L1=300, d2=0.1, L2=30)
    t = tab.d1
    c = tab.coef[:299]
    f, e, d, cc, b, a = (c[..., k] for k in range(6))
    g = ((((a * t + b) * t + cc) * t + d) * t + e) * t + f
    g1 = (((5 * a * t + 4 * b) * t + 3 * cc) * t + 2 * d) * t + e
    g2 = ((20 * a * t + 12 * b) * t + 6 * cc) * t + 2 * d
    xs = np.array([-0.6 + l * 0.01 for l in range(1, 300)])
    y, dy, d2y = embed_d2(xs, net)
    np.testing.assert_allclose(g, y, rtol=0, atol=1e-13)
    np.testing.assert_allclose(g1, dy, rtol=0, atol=1e-10)
    np.testing.assert_allclose(g2, d2y, rtol=0, atol=1e-7)


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_tabulation_error_main_range(seed):
    # brute force against the un-tabulated net: |g - G| <= 1e-9 at stride 0.01
    net = random_net(np.random.default_rng(seed), (1, 25, 50, 100))
    tab = build_table(net, lo=-0.8, d1=0.01, L1=520, d2=0.1, L2=52)
    x = np.random.default_rng(100 + seed).uniform(-0.8, tab.x_up, 20000)
    g, g1 = tab.evaluate(x)
    G, dG, _ = embed_d2(x, net)
    assert np.max(np.abs(g - G)) <= 1e-9
    assert np.max(np.abs(g1 - dG)) <= 1e-6


def test_tabulation_error_band_and_order():
    # band (stride 0.1) is looser; halving the stride divides the error by
    # about 2^6 = 64 (quintic Hermite interpolation is sixth order)
    net = random_net(np.random.default_rng(11), (1, 25, 50, 100))
    tab = build_table(net, lo=-0.8, d1=0.01, L1=400, d2=0.1, L2=40)
    xb = np.random.default_rng(3).uniform(tab.x_up, tab.x_end - 1e-12, 20000)
    assert np.max(np.abs(tab.evaluate(xb)[0] - embed(xb, net))) <= 1e-7
    errs = []
    for dt in (0.08, 0.04, 0.02):
        L = int(round(3.2 / dt))
        t2 = build_table(net, lo=-0.8, d1=dt, L1=L, d2=0.1, L2=1)
        x = np.random.default_rng(4).uniform(-0.8, -0.8 + 3.2, 40000)
        errs.append(np.max(np.abs(t2.evaluate(x)[0] - embed(x, net))))
    r1, r2 = errs[0] / errs[1], errs[1] / errs[2]
    assert 30 < r1 < 130 and 30 < r2 < 130, errs


def test_locate_rules():
    net = random_net(np.random.default_rng(2), (1, 4, 8, 16))
    tab = build_table(net, lo=-0.5, d1=0.01, L1=100, d2=0.1, L2=10)
    # exactly on a node: t = 0 and g = G(node) exactly (f = y_l)
    xn = np.array([-0.5 + l * 0.01 for l in (0, 13, 99)])
    l, t, cl = tab.locate(xn)
    assert list(l) == [0, 13, 99] and np.all(t == 0) and not cl.any()
    np.testing.assert_array_equal(tab.evaluate(xn)[0], embed(xn, net))
    # below lo: interval 0, negative offset
    l, t, cl = tab.locate(np.array([-0.6]))
    assert l[0] == 0 and abs(t[0] + 0.1) < 1e-15 and not cl[0]
    # band and beyond
    l, t, cl = tab.locate(np.array([tab.x_up + 0.25, tab.x_end + 3.0]))
    assert l[0] == 102 and abs(t[0] - 0.05) < 1e-12 and l[1] == 109 and cl[1]
    g, g1 = tab.evaluate(np.array([tab.x_end + 3.0, tab.x_end + 50.0]))
    np.testing.assert_allclose(g[0], embed(np.array([tab.x_end]), net)[0], atol=1e-10)
    assert np.all(g1 == 0) and np.all(g[0] == g[1])


def test_table_memory_inverse_stride():
    # paper hyper-parameter note (4): table memory grows as 1/stride
    net = random_net(np.random.default_rng(2), (1, 4, 8, 16))
    n1 = build_table(net, -0.5, 0.01, 300, 0.1, 1).coef.nbytes
    n2 = build_table(net, -0.5, 0.001, 3000, 0.1, 1).coef.nbytes
    assert abs(n2 / n1 - 10) < 0.05
