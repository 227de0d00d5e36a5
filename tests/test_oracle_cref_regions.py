"""The C oracle's interval location in every part of the tabulated range.

The kernels' band and clamp paths are checked against the C oracle, so its
``locate`` must itself be pinned in all four parts (paper Sec. II: equal
steps over [s^(r_c), s^(r_l)]; the band and the clamp are a reading where
the paper is silent): below the lower end (interval 0, t < 0), the main range, the
extrapolation band and past its end (clamped: value at the end, zero
derivative).  The numpy oracle's ``Table.locate`` is pinned on its own
(closed forms, tabulation error in the band, the locate rules); here the C
oracle must agree with it to rounding on inputs in all four parts, and
copies of the C oracle with a planted mistake in one branch must not.
"""
import os

import numpy as np
import pytest

from oracle import cref
from oracle.se_a import backward, forward
from oracle.table import build_tables
from synth.edge import SHARES, edge_inputs, place_x

from parity import normwise

SRC = os.path.join(os.path.dirname(cref.__file__), "se_a_ref.c")

# one planted mistake per branch of locate(): (original text, replacement)
MUTATIONS = {
    "band uses the main stride": ("floor((x - x_up) / d2)", "floor((x - x_up) / d1)"),
    "band offset from the wrong node": ("*t = x - (x_up + q * d2);", "*t = x - (x_up + (q + 1) * d2);"),
    "clamp offset is not the band stride": ("*t = d2;", "*t = 0.0;"),
    "clamp keeps the derivative": ("double gp = cl ? 0.0", "double gp = 0 ? 0.0"),
    "below lo not clamped to interval 0": ("if (q < 0) q = 0;\n    if (q > (double)(L1 - 1))",
                                           "if (q < 0) q = q;\n    if (q > (double)(L1 - 1))"),
    "band index not clamped": ("if (q > (double)(L2 - 1)) q = (double)(L2 - 1);", ""),
}


def _inputs(seed=0):
    # 40 atoms, two types (4 pairs), every slot valid half the time
    return edge_inputs(40, (30, 50), 24, 8, seed=seed, lo=-0.6, L1=120, L2=12, fill=0.5)


def _compare(x, pb):
    tabs = build_tables(x)
    T0, D0 = forward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2)
    dR0 = backward(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.dT)
    T, D = pb.forward()
    dR = pb.backward(x.dT)
    return max(normwise(T, T0), normwise(D, D0), normwise(dR, dR0))


def _problem(x, lib=None):
    tabs = build_tables(x)
    if lib is not None:
        # a planted mistake may index one interval past the last pair's table:
        # an unused table of NaNs after it keeps that read inside the buffer
        last = tabs[-1]
        tabs = tabs + [type(last)(last.lo, last.d1, last.L1, last.d2, last.L2,
                                  np.full_like(last.coef, np.nan))]
    return cref.Problem(x.em, x.nlist, x.atype, tabs, x.cfg.sel, x.cfg.m2, lib=lib)


def test_inputs_cover_every_part():
    x = _inputs()
    lo, d1, L1, d2, L2 = x.lo[0], x.cfg.d1, int(x.L1[0]), x.cfg.d2, int(x.L2[0])
    x_up, x_end = lo + L1 * d1, lo + L1 * d1 + L2 * d2
    s = x.em[..., 0][x.nlist >= 0]
    n = len(s)
    parts = [(s < lo), (s >= lo) & (s < x_up), (s >= x_up) & (s < x_end), (s >= x_end)]
    for share, p in zip(SHARES, parts):
        assert p.sum() >= 0.8 * share * n
    for v in (lo, x_up, x_end, np.nextafter(x_end, -np.inf)):
        assert np.any(s == v)
    # place_x keeps the shares at any size
    v = place_x(np.random.default_rng(1), 1000, lo, d1, L1, d2, L2)
    assert np.sum(v < lo) == 50 and np.sum(v >= x_end) >= 100


@pytest.mark.parametrize("seed", [0, 1])
def test_c_oracle_matches_numpy_oracle_in_every_part(seed):
    x = _inputs(seed)
    assert _compare(x, _problem(x)) <= 1e-13


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_locate_mistakes_are_caught(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    bad = tmp_path / "se_a_ref_bad.c"
    bad.write_text(src.replace(old, new))
    lib = cref.load_library(cref.compile_source(str(bad), str(tmp_path / "libbad.so")))
    x = _inputs()
    err = _compare(x, _problem(x, lib))
    assert not err <= 1e-6, name      # NaN (an interval past the table) also fails
