"""GPU neighbour list (dpc_nlist_build) against the brute-force oracle.

Integer output: bit-exact against oracle/nlist_ref.c (same distance formula,
same order (type, r^2, index)) on every atom of the small workloads and on
sampled atoms of the 1,048,576-atom one; against the generator's lists the
sets per type block are equal and the order agrees up to exact distance
ties (water's rigid oxygens on a grid)."""
import numpy as np
import pytest

from oracle import nlist as onl
from synth import make_inputs
from synth.configs import get_config

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

_CACHE = {}


def _inputs(key):
    if key not in _CACHE:
        _CACHE.clear()
        print(f"[gpu-nlist] generating {key}", flush=True)
        _CACHE[key] = make_inputs(get_config(key), with_grad=False)
    return _CACHE[key]


def _gpu(coord, atype, sel, box, rc, wait=True, ws_extra=0):
    import paper_2107_02103_amd as P
    n = len(coord)
    c = torch.from_numpy(np.ascontiguousarray(coord, np.float64)).cuda()
    a = torch.from_numpy(np.ascontiguousarray(atype, np.int32)).cuda()
    nb = P.dpc_nlist_workspace_bytes(n, box, rc)
    ws = torch.empty(nb + ws_extra, dtype=torch.uint8, device="cuda")
    nl = torch.full((n, int(sum(sel))), -7, dtype=torch.int32, device="cuda")
    st = P.dpc_nlist_build(torch.cuda.current_stream(), n, len(sel), sel, box, rc, c, a, ws, nb, nl,
                           wait=wait)
    torch.cuda.synchronize()
    if not wait:
        st = tuple(ws[:8].view(torch.int32).cpu().tolist())
    return nl.cpu().numpy(), st


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water", 0, 1, 2])
def test_bit_exact_all_atoms(key):
    x = _inputs(key)
    c = x.cfg
    got, st = _gpu(x.coords, x.atype, c.sel, c.box, c.rc)
    ref, cnt, over = onl.neighbour_list(x.coords, x.atype, c.sel, c.box, c.rc)
    print(f"[gpu-nlist] {c.name}: {len(got)} atoms, status {st}, "
          f"{int((got >= 0).sum())} neighbours", flush=True)
    assert st == (0, 0) and over == 0
    np.testing.assert_array_equal(got, ref)
    if c.kind == "fcc":        # no exact ties: the generator's lists too
        np.testing.assert_array_equal(got, x.nlist)
    else:
        for i in range(len(got)):
            assert set(got[i][got[i] >= 0]) == set(x.nlist[i][x.nlist[i] >= 0])


@pytest.mark.timeout(600)
def test_cu1m_sampled():
    # the benchmarked workload: 1,048,576 atoms, sel 512, r_c 8
    x = _inputs(3)
    c = x.cfg
    got, st = _gpu(x.coords, x.atype, c.sel, c.box, c.rc)
    assert st == (0, 0)
    atoms = np.unique(np.concatenate([np.random.default_rng(5).choice(len(got), 400, replace=False),
                                      [0, len(got) - 1]]))
    ref, cnt, over = onl.neighbour_list(x.coords, x.atype, c.sel, c.box, c.rc, centres=atoms)
    print(f"[gpu-nlist] cu1m: {len(atoms)} sampled atoms, {int((ref >= 0).sum())} neighbours", flush=True)
    assert over == 0
    np.testing.assert_array_equal(got[atoms], ref)
    # the generator's lists of every atom (jittered crystal: no exact ties)
    np.testing.assert_array_equal(got, x.nlist)


def test_truncation_reports_overflow():
    import paper_2107_02103_amd as P
    x = _inputs("tiny_alloy")
    c = x.cfg
    small = (10, 3, 3)
    with pytest.raises(P.DpcError) as e:
        _gpu(x.coords, x.atype, small, c.box, c.rc)
    assert e.value.status == P.DPC_EOVERFLOW
    got, st = _gpu(x.coords, x.atype, small, c.box, c.rc, wait=False)
    ref, cnt, over = onl.neighbour_list(x.coords, x.atype, small, c.box, c.rc)
    assert over > 0 and st == (over, 0)
    np.testing.assert_array_equal(got, ref)


def test_positions_outside_the_box_and_shuffled_atoms():
    x = _inputs("tiny_water")
    c = x.cfg
    rng = np.random.default_rng(3)
    shifted = x.coords + c.box * rng.integers(-3, 4, size=x.coords.shape)
    got, _ = _gpu(shifted, x.atype, c.sel, c.box, c.rc)
    ref, _, _ = onl.neighbour_list(shifted, x.atype, c.sel, c.box, c.rc)
    np.testing.assert_array_equal(got, ref)
    perm = rng.permutation(len(x.coords))
    got, _ = _gpu(x.coords[perm], x.atype[perm], c.sel, c.box, c.rc)
    ref, _, _ = onl.neighbour_list(x.coords[perm], x.atype[perm], c.sel, c.box, c.rc)
    np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("edge", [2.0000000001, 2.05, 2.6, 3.5])
def test_few_cells_per_edge(edge):
    # box / r_c just above 2 (1 or 2 cells per edge) and 3 cells: every
    # stencil shape; random positions and three types, one of them invalid
    rng = np.random.default_rng(int(edge * 100))
    rc, n = 3.0, 300
    box = edge * rc
    coord = rng.uniform(-box, 2 * box, size=(n, 3))
    atype = rng.integers(-1, 3, size=n).astype(np.int32)
    sel = (120, 120)
    got, st = _gpu(coord, atype, sel, box, rc, wait=False)
    ref, cnt, over = onl.neighbour_list(coord, atype, sel, box, rc)
    assert st == (over, 0)
    np.testing.assert_array_equal(got, ref)


def test_capacity_overflow_is_reported():
    # more than 1024 atoms within r_c of one atom: DPC_ENOTSUP
    import paper_2107_02103_amd as P
    rng = np.random.default_rng(1)
    coord = rng.uniform(0, 4.0, size=(1100, 3))
    with pytest.raises(P.DpcError) as e:
        _gpu(coord, np.zeros(1100, np.int32), (2048,), 100.0, 10.0)
    assert e.value.status == P.DPC_ENOTSUP


def test_deterministic_and_empty():
    import paper_2107_02103_amd as P
    x = _inputs(1)
    c = x.cfg
    a, _ = _gpu(x.coords, x.atype, c.sel, c.box, c.rc)
    b, _ = _gpu(x.coords, x.atype, c.sel, c.box, c.rc)
    np.testing.assert_array_equal(a, b)
    e = torch.zeros((0, 3), dtype=torch.float64, device="cuda")
    t = torch.zeros((0,), dtype=torch.int32, device="cuda")
    nl = torch.zeros((0, 10), dtype=torch.int32, device="cuda")
    ws = torch.zeros(256, dtype=torch.uint8, device="cuda")
    assert P.dpc_nlist_build(0, 0, 1, [10], 20.0, 5.0, e, t, ws, 256, nl) == (0, 0)


def test_half_box_differences():
    # coordinate differences of exactly half a box and one unit in the last
    # place either side: the minimum image's rint(d / box) sits on or next to
    # a tie there, where the kernel takes the quotient from a division
    rng = np.random.default_rng(11)
    box, rc = 20.0, 9.5
    base = rng.uniform(0, box, size=(60, 3))
    half = np.array([0.5 * box, 0.0, 0.0])
    coord = [base]
    for step in (-1, 0, 1):
        shifted = base + half
        shifted[:, 0] = np.nextafter(shifted[:, 0], np.inf * step) if step else shifted[:, 0]
        coord.append(shifted)
    coord.append(base + np.array([0.5 * box, 0.5 * box, -0.5 * box]))
    coord = np.concatenate(coord)
    atype = rng.integers(0, 2, size=len(coord)).astype(np.int32)
    sel = (300, 300)
    got, st = _gpu(coord, atype, sel, box, rc, wait=False)
    ref, cnt, over = onl.neighbour_list(coord, atype, sel, box, rc)
    assert st == (over, 0)
    np.testing.assert_array_equal(got, ref)
