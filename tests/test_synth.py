"""Checks of the synthetic input generator (not part of the method)."""
import numpy as np
import pytest

from synth import make_inputs
from synth.configs import CONFIGS, TEST_CONFIGS, get_config
from synth.system import _rngs, _structure, weighting


def test_weighting_function_eq1():
    rc, rcs = 6.0, 0.5
    r = np.array([0.3, rcs, 2.0, rc - 1e-12, rc, 7.0])
    s = weighting(r, rc, rcs)
    assert s[0] == 1 / 0.3 and s[1] == 1 / rcs          # 1/r inside r_cs, switch = 1 at r_cs
    u = (2.0 - rcs) / (rc - rcs)
    assert abs(s[2] - (u ** 3 * (-6 * u * u + 15 * u - 10) + 1) / 2.0) < 1e-15
    assert abs(s[3]) < 1e-12 and s[4] == 0 and s[5] == 0
    # the switch is C^2 at both ends: first and second derivative vanish
    sw = lambda u: u ** 3 * (-6 * u * u + 15 * u - 10) + 1
    h = 1e-4
    for u0 in (0.0, 1.0):
        assert abs((sw(u0 + h) - sw(u0 - h)) / (2 * h)) < 1e-6
        assert abs((sw(u0 + h) - 2 * sw(u0) + sw(u0 - h)) / h ** 2) < 1e-3


@pytest.mark.parametrize("key", list(TEST_CONFIGS))
def test_neighbour_list_matches_brute_force(key):
    cfg = get_config(key)
    x = make_inputs(cfg)
    rp, rs, ro, *_ = _rngs(cfg)
    basis, types, disp = _structure(cfg, rp, rs, ro)
    N, L, nb = cfg.ncell, cfg.cell_edge, len(basis)
    cells = np.arange(N ** 3)
    cpos = np.stack([cells // (N * N), (cells // N) % N, cells % N], 1) * L
    pos = (cpos[:, None, :] + basis[None]).reshape(-1, 3) + disp
    box = cfg.box
    off = np.concatenate([[0], np.cumsum(cfg.sel)])
    for i in range(len(pos)):
        d = pos - pos[i]
        d -= box * np.round(d / box)
        r = np.linalg.norm(d, axis=1)
        r[i] = np.inf
        for b in range(cfg.ntypes):
            want = np.nonzero((r < cfg.rc) & (types == b))[0]
            want = want[np.argsort(r[want], kind="stable")]
            blk = x.nlist[i, off[b]:off[b + 1]]
            got = blk[blk >= 0]
            assert sorted(got) == sorted(want)
            np.testing.assert_allclose(r[got], np.sort(r[want]), atol=1e-12)   # distance sorted
            assert np.all(blk[len(got):] == -1)                               # padding at the end


def test_normalisation_and_padding():
    x = make_inputs(get_config("tiny_water"))
    v = x.nlist >= 0
    assert np.all(x.em[~v] == 0)
    for a in range(x.cfg.ntypes):
        rows = v & (x.atype[:, None] == a)
        s = x.em[rows][:, 0]
        assert abs(s.mean()) < 1e-12 and abs(s.std() - 1) < 1e-12
        xyz = x.em[rows][:, 1:].ravel()
        assert abs(xyz.std() - 1) < 1e-2        # pooled sigma_all (mean not removed)
    # table range covers every observed s^ with a margin below one interval
    for a in range(2):
        for b in range(2):
            p = a * 2 + b
            assert x.lo[p] + x.L1[p] * x.d1 > x.s_hat_max[p] >= x.lo[p] + (x.L1[p] - 1) * x.d1


def test_deterministic_and_thread_independent():
    c = get_config("tiny_alloy")
    a = make_inputs(c, threads=1, chunk_cells=5)
    b = make_inputs(c, threads=4, chunk_cells=5)
    np.testing.assert_array_equal(a.em, b.em)
    np.testing.assert_array_equal(a.nlist, b.nlist)
    np.testing.assert_array_equal(a.dT, b.dT)


def test_config_shapes():
    assert [c.natoms for c in CONFIGS] == [256, 12288, 32000, 1048576, 331776]
    assert [c.nnei for c in CONFIGS] == [128, 138, 420, 512, 138]
    assert abs(get_config("water4096").box - 49.669) < 1e-3 and abs(get_config("water110592").box - 149.0) < 0.01
