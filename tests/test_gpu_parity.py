"""GPU parity: the HIP kernels (through the C ABI) against the oracle on the
same seeded inputs.  fp64 to 1e-12 and fp32 / mixed modes to 1e-5, per-atom
normwise and abs-sum-scaled componentwise."""
import numpy as np
import pytest

from synth import make_inputs
from synth.configs import get_config

from parity import TOL, compare, oracle_abs_bounds, oracle_fwd_bwd

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

_CACHE = {}


def _inputs(key):
    if key not in _CACHE:
        _CACHE.clear()          # keep at most one big config resident
        print(f"[gpu-parity] generating {key}", flush=True)
        _CACHE[key] = make_inputs(get_config(key))
    return _CACHE[key]


def _mode(dtype):
    import paper_2107_02103_amd as P
    return {"f64": (P.DPC_F64, np.float64), "f32": (P.DPC_F32, np.float32),
            "f32acc64": (P.DPC_F32_ACC64, np.float32)}[dtype]


def _run_gpu(x, dtype="f64"):
    import paper_2107_02103_amd as P
    mode, store = _mode(dtype)
    c = x.cfg
    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, c.d1, c.d2, c.sel, c.m2, dtype=mode)
    dev = "cuda"
    em = torch.from_numpy(x.em.astype(store, copy=False)).to(dev)
    nl = torch.from_numpy(x.nlist).to(dev)
    at = torch.from_numpy(x.atype).to(dev)
    dT = torch.from_numpy(x.dT.astype(store, copy=False)).to(dev)
    T, D = op.forward(em, nl, at)
    dR = op.backward(em, nl, at, dT)
    torch.cuda.synchronize()
    return op, (em, nl, at, dT), (T, D, dR)


def _check(x, atoms, got, dtype, with_bounds=True):
    tol = TOL[dtype]
    ref = oracle_fwd_bwd(x, atoms, dtype)
    bounds = oracle_abs_bounds(x, atoms, dtype) if with_bounds else None
    g = tuple(a[atoms] for a in got)
    rep = compare(g, ref, bounds, tol)
    print(f"[gpu-parity] {x.cfg.name} {dtype} atoms={len(atoms)} {rep}", flush=True)
    assert rep["ok"], rep
    # padding rows of dE/dR~ are exactly zero
    assert np.all(g[2][x.nlist[atoms] < 0] == 0)


def _sample(n, k, seed=0):
    rng = np.random.default_rng(seed)
    s = rng.choice(n, size=min(k, n), replace=False)
    return np.unique(np.concatenate([s, [0, n - 1]]))


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water", 0, 1, 2])
def test_parity_f64(key):
    x = _inputs(key)
    _, _, out = _run_gpu(x, "f64")
    got = tuple(t.cpu().numpy() for t in out)
    n = x.nlist.shape[0]
    # every atom normwise against the C oracle, a sample componentwise
    ref = oracle_fwd_bwd(x, np.arange(n), "f64")
    rep = compare(got, ref, None, TOL["f64"])
    print(f"[gpu-parity] {x.cfg.name} all atoms {rep}", flush=True)
    assert rep["ok"], rep
    _check(x, _sample(n, 300), got, "f64")


def _all_atoms_normwise(x, out, dtype, chunk=65536):
    """Every atom's T, D and dE/dR~ normwise against the C oracle, in chunks
    of atoms (the oracle's tables are built once)."""
    from oracle import cref
    from parity import normwise, oracle_view
    tabs, em, nl, at, dT = oracle_view(x, slice(None), dtype)
    pb = cref.Problem(em, nl, at, tabs, x.cfg.sel, x.cfg.m2)
    n = nl.shape[0]
    worst = {"T": 0.0, "D": 0.0, "dR": 0.0}
    for a0 in range(0, n, chunk):
        a1 = min(n, a0 + chunk)
        T, D = pb.forward(a0, a1)
        dR = pb.backward(dT[a0:a1], a0, a1)
        for name, g, r in zip(("T", "D", "dR"), out, (T, D, dR)):
            worst[name] = max(worst[name], normwise(g[a0:a1].cpu().numpy().astype(np.float64), r))
        # padding rows of dE/dR~ are exactly zero
        assert np.all(out[2][a0:a1].cpu().numpy()[nl[a0:a1] < 0] == 0)
    print(f"[gpu-parity] {x.cfg.name} {dtype} all {n} atoms normwise {worst}", flush=True)
    assert max(worst.values()) <= TOL[dtype], worst


@pytest.mark.timeout(900)
def test_parity_f64_full_size_cu1m():
    # the benchmarked workload (1,048,576 atoms, sel 512): every atom
    # normwise, a sample componentwise
    x = _inputs(3)
    _, _, out = _run_gpu(x, "f64")
    _all_atoms_normwise(x, out, "f64")
    atoms = _sample(x.nlist.shape[0], 400, seed=3)
    got = tuple(t[torch.from_numpy(atoms).cuda()].cpu().numpy() for t in out)
    tol = TOL["f64"]
    ref = oracle_fwd_bwd(x, atoms, "f64")
    bounds = oracle_abs_bounds(x, atoms, "f64")
    rep = compare(got, ref, bounds, tol)
    print(f"[gpu-parity] cu1m sampled {rep}", flush=True)
    assert rep["ok"], rep
    del out
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("dtype", ["f32", "f32acc64", "f64"])
def test_parity_water_large_modes(dtype):
    # water110592 (331,776 atoms) in all three modes: every atom normwise, a
    # sample componentwise
    x = _inputs(4)
    _, _, out = _run_gpu(x, dtype)
    _all_atoms_normwise(x, out, dtype)
    atoms = _sample(x.nlist.shape[0], 300, seed=4)
    got = tuple(t[torch.from_numpy(atoms).cuda()].cpu().numpy().astype(np.float64) for t in out)
    tol = TOL[dtype]
    rep = compare(got, oracle_fwd_bwd(x, atoms, dtype), oracle_abs_bounds(x, atoms, dtype), tol)
    print(f"[gpu-parity] water110592 {dtype} sampled {rep}", flush=True)
    assert rep["ok"], rep


@pytest.mark.parametrize("dtype", ["f32", "f32acc64"])
def test_parity_small_fp32_modes(dtype):
    x = _inputs(1)
    _, _, out = _run_gpu(x, dtype)
    got = tuple(t.cpu().numpy().astype(np.float64) for t in out)
    _check(x, _sample(x.nlist.shape[0], 300, seed=1), got, dtype)


def test_deterministic_bitwise():
    x = _inputs(2)
    op, (em, nl, at, dT), out1 = _run_gpu(x, "f64")
    T2, D2 = op.forward(em, nl, at)
    dR2 = op.backward(em, nl, at, dT)
    torch.cuda.synchronize()
    assert torch.equal(out1[0], T2) and torch.equal(out1[1], D2) and torch.equal(out1[2], dR2)


def _synthetic(nloc, sel, m1, m2, seed, **kw):
    """Hand-placed rows in every part of the tabulated range (below lo, main
    range, band, past the band; fixed shares) for edge cases."""
    from synth.edge import edge_inputs
    return edge_inputs(nloc, sel, m1, m2, seed, **kw)


@pytest.mark.parametrize("sel,m1,m2", [((3, 70), 100, 16), ((64,), 64, 64), ((5, 1, 60), 200, 7),
                                       ((130,), 1, 1), ((1,), 100, 100),
                                       # more slots than one window of nlist signs (512 or
                                       # 1024 per atom), ragged at the end
                                       ((700, 900), 100, 16), ((2100,), 64, 16),
                                       # K steps of the float64 matrix-core backward: odd
                                       # and even per channel quarter, its largest M1 and
                                       # the first M1 past it
                                       ((77,), 17, 4), ((40, 33), 128, 16), ((20,), 113, 16),
                                       ((50,), 129, 8)])
def test_edge_shapes_and_ranges(sel, m1, m2):
    # ragged nnei, m1 not a multiple of 64 (and m1 > 128), m2 = m1, a single
    # channel, inputs below lo and beyond the band (clamped), empty atoms
    x = _synthetic(37, sel, m1, m2, seed=sum(sel) + m1)
    x.nlist[5] = -1
    x.em[5] = 0
    _, _, out = _run_gpu(x, "f64")
    got = tuple(t.cpu().numpy() for t in out)
    _check(x, np.arange(37), got, "f64")
    assert np.all(got[0][5] == 0) and np.all(got[1][5] == 0) and np.all(got[2][5] == 0)


@pytest.mark.parametrize("dtype", ["f32acc64", "f32"])
@pytest.mark.parametrize("sel,m1,m2", [((3, 70), 100, 16), ((77,), 17, 4), ((40, 33), 128, 16),
                                       ((20,), 113, 16), ((50,), 129, 8), ((700, 900), 100, 16)])
def test_edge_shapes_float32_modes(sel, m1, m2, dtype):
    # the mixed mode's backward on the matrix cores (float32 tables copied
    # into LDS, 8 bytes per power pair) and the float32 vector kernels
    x = _synthetic(37, sel, m1, m2, seed=sum(sel) + m1 + 7)
    x.nlist[5] = -1
    x.em[5] = 0
    _, _, out = _run_gpu(x, dtype)
    got = tuple(t.cpu().numpy().astype(np.float64) for t in out)
    _check(x, np.arange(37), got, dtype)


def test_empty_and_single_atom():
    import paper_2107_02103_amd as P
    x = _synthetic(1, (40,), 100, 16, seed=3)
    _, _, out = _run_gpu(x, "f64")
    _check(x, np.arange(1), tuple(t.cpu().numpy() for t in out), "f64")
    c = x.cfg
    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, c.d1, c.d2, c.sel, c.m2)
    e = torch.zeros((0, 40, 4), dtype=torch.float64, device="cuda")
    nl = torch.zeros((0, 40), dtype=torch.int32, device="cuda")
    at = torch.zeros((0,), dtype=torch.int32, device="cuda")
    T, D = op.forward(e, nl, at)
    dR = op.backward(e, nl, at, torch.zeros((0, 100, 4), dtype=torch.float64, device="cuda"))
    torch.cuda.synchronize()
    assert T.shape == (0, 100, 4) and D.shape == (0, 100, 16) and dR.shape == (0, 40, 4)


@pytest.mark.parametrize("col,val", [(1, np.nan), (0, np.nan), (0, np.inf), (0, -np.inf)])
def test_nan_stays_in_its_atom(col, val):
    # a non-finite entry of R~ makes the same outputs non-finite as in the
    # oracle (a NaN or infinite first column is not silently clamped away)
    # and no other atom's
    x = _synthetic(9, (50,), 100, 16, seed=4)
    j = int(np.nonzero(x.nlist[2] >= 0)[0][0])
    x.em[2, j, col] = val
    _, _, out = _run_gpu(x, "f64")
    T, D, dR = (t.cpu().numpy() for t in out)
    assert not np.isfinite(T[2]).all()
    others = [i for i in range(9) if i != 2]
    assert np.isfinite(T[others]).all() and np.isfinite(D[others]).all() and np.isfinite(dR[others]).all()
    _check(x, np.array(others), (T, D, dR), "f64", with_bounds=False)
    ref = oracle_fwd_bwd(x, np.array([2]), "f64")
    for name, g, r in zip(("T", "D", "dR"), (T[2:3], D[2:3], dR[2:3]), ref):
        np.testing.assert_array_equal(np.isfinite(g), np.isfinite(r), err_msg=name)
        f = np.isfinite(r)
        if f.any():
            assert np.max(np.abs(g[f] - r[f])) <= 1e-12 * np.max(np.abs(r[f])), name


@pytest.mark.parametrize("m1", [100, 17])
def test_coefficients_past_the_buffer_are_not_read(m1):
    # the coefficient tensor is a view into a larger allocation whose tail
    # holds NaN; records in the last interval of the last type pair (clamped
    # ones, a tenth of all) must not pick any of it up
    import paper_2107_02103_amd as P
    x = _synthetic(64, (40, 40), m1, 4, seed=m1)
    c = x.cfg
    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, c.d1, c.d2, c.sel, c.m2)
    n = op.coeff.numel()
    big = torch.full((n + 4096,), float("nan"), dtype=torch.float64, device="cuda")
    big[:n] = op.coeff
    op.coeff = big[:n]
    last = (x.atype == c.ntypes - 1)[:, None] & (np.arange(c.nnei) >= c.sel[0])[None, :]
    x_end = x.lo[-1] + x.L1[-1] * c.d1 + x.L2[-1] * c.d2
    assert np.sum(last & (x.nlist >= 0) & (x.em[..., 0] >= x_end)) > 20
    em = torch.from_numpy(x.em).cuda()
    nl = torch.from_numpy(x.nlist).cuda()
    at = torch.from_numpy(x.atype).cuda()
    dT = torch.from_numpy(x.dT).cuda()
    T, D = op.forward(em, nl, at)
    dR = op.backward(em, nl, at, dT)
    torch.cuda.synchronize()
    got = tuple(t.cpu().numpy() for t in (T, D, dR))
    assert all(np.isfinite(g).all() for g in got)
    _check(x, np.arange(64), got, "f64")


@pytest.mark.parametrize("dtype", ["f64", "f32acc64", "f32"])
def test_mixed_and_invalid_types_in_one_workgroup(dtype):
    # three types in random order, plus atoms of invalid type (-1 and
    # ntypes): a workgroup hands its atoms to its wavefronts grouped by type,
    # invalid ones last; every valid atom still matches the oracle, every
    # invalid one gets NaN outputs, and runs repeat bitwise
    x = _synthetic(77, (30, 20, 14), 100, 16, seed=21)
    rng = np.random.default_rng(5)
    x.atype[:] = rng.integers(0, 3, size=77).astype(np.int32)
    bad = np.array([3, 16, 17, 40, 76])
    x.atype[bad[:3]] = -1
    x.atype[bad[3:]] = 3
    T, D, dR = (t.cpu().numpy() for t in _run_gpu(x, dtype)[2])
    for a in (T, D, dR):
        assert np.isnan(a[bad]).all()
    good = np.setdiff1d(np.arange(77), bad)
    _check(x, good, (T, D, dR), dtype)
    T2, D2, dR2 = (t.cpu().numpy() for t in _run_gpu(x, dtype)[2])
    for a, b in ((T, T2), (D, D2), (dR, dR2)):
        np.testing.assert_array_equal(a[good], b[good])
