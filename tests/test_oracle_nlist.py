"""Pins of the brute-force neighbour-list oracle (oracle/nlist_ref.c).

Paper Sec. II: the neighbours of atom i within r_c, in sel_beta slots per
neighbour type, sorted by distance inside each type block, unused slots
empty.  The oracle is checked against things other than itself: the
seeded generator's lists (built from lattice-site offsets, not from a
search), the shell structure of a perfect fcc crystal, the symmetry of the
relation, the nearest-first truncation rule, and copies with planted
mistakes."""
import os

import numpy as np
import pytest

from oracle import nlist as onl
from synth import make_inputs
from synth.configs import get_config


def _dist2(coord, box, i, js):
    d = coord[js] - coord[i]
    d -= box * np.rint(d / box)
    return (d * d).sum(-1)


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water", 0, 1])
def test_matches_generator(key):
    # the generator takes the sites within r_c (+ displacement bound) from a
    # fixed list of lattice offsets and sorts them; equal distances (water's
    # rigid oxygens on a grid) may come in another order there
    x = make_inputs(get_config(key))
    c = x.cfg
    nl, cnt, over = onl.neighbour_list(x.coords, x.atype, c.sel, c.box, c.rc)
    assert over == 0
    off = np.concatenate([[0], np.cumsum(c.sel)])
    for i in range(len(nl)):
        for b in range(c.ntypes):
            a = nl[i, off[b]:off[b + 1]]
            g = x.nlist[i, off[b]:off[b + 1]]
            assert np.array_equal(a < 0, g < 0)
            a, g = a[a >= 0], g[g >= 0]
            assert set(a) == set(g)
            assert cnt[i, b] == len(a)
            if not np.array_equal(a, g):
                da, dg = _dist2(x.coords, c.box, i, a), _dist2(x.coords, c.box, i, g)
                assert np.allclose(da, dg, rtol=1e-12, atol=0)
    if get_config(key).kind == "fcc":
        assert np.array_equal(nl, x.nlist)


def test_fcc_shells():
    # perfect fcc crystal (no jitter), a = 3.634, r_c between the third
    # (a sqrt(3/2), 24 sites) and the fourth shell (a sqrt(2)): 12 + 6 + 24
    # neighbours at a / sqrt(2), a and a sqrt(3/2), in that order
    a, n = 3.634, 4
    basis = a * np.array([[0, 0, 0], [0.5, 0.5, 0], [0.5, 0, 0.5], [0, 0.5, 0.5]])
    cells = np.stack(np.meshgrid(*[np.arange(n)] * 3, indexing="ij"), -1).reshape(-1, 3) * a
    coord = (cells[:, None, :] + basis[None]).reshape(-1, 3)
    box, rc = n * a, 4.6
    nl, cnt, over = onl.neighbour_list(coord, np.zeros(len(coord), np.int32), [48], box, rc)
    assert over == 0 and np.all(cnt[:, 0] == 42) and np.all(nl[:, 42:] == -1)
    shells = np.array([a / np.sqrt(2)] * 12 + [a] * 6 + [a * np.sqrt(1.5)] * 24)
    for i in (0, 1, 77, len(coord) - 1):
        d = np.sqrt(_dist2(coord, box, i, nl[i, :42]))
        np.testing.assert_allclose(d, shells, rtol=1e-12)
        # exactly equal squared distances come in ascending index order
        r2 = _dist2(coord, box, i, nl[i, :42])
        assert np.all(np.diff(r2) >= 0)
        tie = np.diff(r2) == 0
        assert np.all(np.diff(nl[i, :42])[tie] > 0) and tie.any()


def test_symmetric_and_within_cutoff():
    x = make_inputs(get_config("tiny_alloy"))
    c = x.cfg
    nl, _, _ = onl.neighbour_list(x.coords, x.atype, c.sel, c.box, c.rc)
    pairs = {(i, int(j)) for i in range(len(nl)) for j in nl[i] if j >= 0}
    assert all((j, i) in pairs for i, j in pairs)
    for i, j in list(pairs)[:500]:
        assert _dist2(x.coords, c.box, i, np.array([j]))[0] < c.rc ** 2


def test_truncation_keeps_the_nearest():
    x = make_inputs(get_config("tiny_alloy"))
    c = x.cfg
    full, cnt, _ = onl.neighbour_list(x.coords, x.atype, c.sel, c.box, c.rc)
    small = (10, 3, 3)
    nl, cnt2, over = onl.neighbour_list(x.coords, x.atype, small, c.box, c.rc)
    assert np.array_equal(cnt, cnt2)
    assert over == int(np.sum(np.any(cnt > np.array(small), 1)))
    off, off2 = np.concatenate([[0], np.cumsum(c.sel)]), np.concatenate([[0], np.cumsum(small)])
    for i in range(len(nl)):
        for b in range(c.ntypes):
            k = min(small[b], cnt[i, b])
            assert np.array_equal(nl[i, off2[b]:off2[b] + k], full[i, off[b]:off[b] + k])
            assert np.all(nl[i, off2[b] + k:off2[b + 1]] == -1)


def test_exact_cutoff_is_excluded():
    # r^2 == rc^2 exactly (3^2 in binary): not a neighbour
    coord = np.array([[0.0, 0.0, 0.0], [3.0, 0.0, 0.0], [0.0, 2.5, 0.0]])
    nl, cnt, _ = onl.neighbour_list(coord, np.zeros(3, np.int32), [4], 10.0, 3.0)
    assert list(nl[0]) == [2, -1, -1, -1] and list(nl[1]) == [-1] * 4


MUTATIONS = {
    "no minimum image": ("return d - box * rint(d / box);", "return d;"),
    "cutoff inclusive": ("if (r2 < rc2) {", "if (r2 <= rc2) {"),
    "farthest first": ("if (a->r2 != b->r2) return a->r2 < b->r2;", "if (a->r2 != b->r2) return a->r2 > b->r2;"),
    "ties by descending index": ("return a->j < b->j;", "return a->j > b->j;"),
    "blocks in the wrong place": ("for (int q = 0; q < b; ++q) start += sel[q];",
                                  "for (int q = b + 1; q < ntypes; ++q) start += sel[q];"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistakes_are_caught(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(onl.SRC).read()
    assert src.count(old) == 1, name
    bad = tmp_path / "bad.c"
    bad.write_text(src.replace(old, new))
    lib = onl.load_library(onl.compile_source(str(bad), str(tmp_path / "libbad.so")))
    caught = False
    # the shell crystal (ties, periodic images, blocks of one type)
    a, n = 3.634, 4
    basis = a * np.array([[0, 0, 0], [0.5, 0.5, 0], [0.5, 0, 0.5], [0, 0.5, 0.5]])
    cells = np.stack(np.meshgrid(*[np.arange(n)] * 3, indexing="ij"), -1).reshape(-1, 3) * a
    coord = (cells[:, None, :] + basis[None]).reshape(-1, 3)
    good = onl.neighbour_list(coord, np.zeros(len(coord), np.int32), [48], n * a, 4.6)[0]
    caught |= not np.array_equal(good, onl.neighbour_list(coord, np.zeros(len(coord), np.int32), [48],
                                                          n * a, 4.6, lib=lib)[0])
    # the exact cutoff
    c3 = np.array([[0.0, 0.0, 0.0], [3.0, 0.0, 0.0], [0.0, 2.5, 0.0]])
    caught |= not np.array_equal(onl.neighbour_list(c3, np.zeros(3, np.int32), [4], 10.0, 3.0)[0],
                                 onl.neighbour_list(c3, np.zeros(3, np.int32), [4], 10.0, 3.0, lib=lib)[0])
    # three types against the generator
    x = make_inputs(get_config("tiny_alloy"))
    c = x.cfg
    caught |= not np.array_equal(x.nlist, onl.neighbour_list(x.coords, x.atype, c.sel, c.box, c.rc,
                                                             lib=lib)[0])
    assert caught, name
