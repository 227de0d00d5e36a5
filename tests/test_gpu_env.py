"""GPU parity of the environment matrix, the reverse neighbour slots and the
force / virial assembly (through the C ABI) against the oracle, on the
seeded synthetic systems."""
import numpy as np
import pytest

import oracle.env as ev
from synth import make_inputs
from synth.configs import get_config
from synth.system import random_grad

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

_CACHE = {}


def _inputs(key):
    if key not in _CACHE:
        _CACHE.clear()
        print(f"[gpu-env] generating {key}", flush=True)
        _CACHE[key] = make_inputs(get_config(key))
    return _CACHE[key]


def _stats(x):
    s = x.stats
    return s["mean"], s["sigma"], s["sigma_all"]


def _dev(x):
    return (torch.from_numpy(x.coords).cuda(), torch.from_numpy(x.atype).cuda(),
            torch.from_numpy(x.nlist).cuda())


def _env_gpu(x, dtype="f64"):
    import paper_2107_02103_amd as P
    c = x.cfg
    mode = {"f64": P.DPC_F64, "f32": P.DPC_F32}[dtype]
    coord, at, nl = _dev(x)
    em = torch.full((len(x.atype), c.nnei, 4), float("nan"),
                    dtype=torch.float64 if dtype == "f64" else torch.float32, device="cuda")
    P.dpc_env_mat_a(torch.cuda.current_stream(), mode, len(x.atype), c.ntypes, c.nnei, c.box, c.rc,
                    c.rcs, *_stats(x), coord, at, nl, em)
    torch.cuda.synchronize()
    return em.cpu().numpy().astype(np.float64)


def _normwise(g, r):
    den = np.maximum(np.abs(r).reshape(len(r), -1).max(1), 1e-300)
    return float(np.max(np.abs(g - r).reshape(len(r), -1).max(1) / den))


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water", 0, 1])
def test_env_mat_parity(key):
    x = _inputs(key)
    c = x.cfg
    em = _env_gpu(x)
    ref = ev.env_mat(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, *_stats(x))
    err = _normwise(em, ref)
    print(f"[gpu-env] {c.name} env_mat normwise {err:.2e}", flush=True)
    assert err <= 1e-12
    assert np.all(em[x.nlist < 0] == 0)
    # the same rows as the generator's own R~
    assert _normwise(em, x.em) <= 1e-12
    # float32 output: the float64 rows rounded
    em32 = _env_gpu(x, "f32")
    assert np.array_equal(em32, em.astype(np.float32).astype(np.float64))


@pytest.mark.timeout(600)
def test_env_mat_full_size_cu1m_sampled():
    x = _inputs(3)
    c = x.cfg
    em = _env_gpu(x)
    atoms = np.unique(np.concatenate([np.random.default_rng(6).choice(len(x.atype), 60, replace=False),
                                      [0, len(x.atype) - 1]]))
    ref = ev.env_mat(x.coords, c.box, x.atype[atoms], x.nlist[atoms], c.rc, c.rcs, *_stats(x), atoms=atoms)
    err = _normwise(em[atoms], ref)
    print(f"[gpu-env] cu1m env_mat sampled normwise {err:.2e}", flush=True)
    assert err <= 1e-12
    assert np.all(em[x.nlist < 0] == 0)


def _reverse_expected(nlist, atype, sel):
    off = np.concatenate([[0], np.cumsum(sel)])
    n, nnei = nlist.shape
    rev = np.full((n, nnei), -1, np.int32)
    for i in range(n):
        for s in np.nonzero(nlist[i] >= 0)[0]:
            j = nlist[i, s]
            t = atype[i]
            hit = np.nonzero(nlist[j, off[t]:off[t + 1]] == i)[0]
            if len(hit):
                rev[i, s] = off[t] + hit[0]
    return rev


def _reverse_gpu(x):
    import paper_2107_02103_amd as P
    c = x.cfg
    coord, at, nl = _dev(x)
    rev = torch.full(x.nlist.shape, -7, dtype=torch.int32, device="cuda")
    P.dpc_nlist_reverse(torch.cuda.current_stream(), len(x.atype), c.ntypes, c.sel, c.box, coord, at,
                        nl, rev)
    torch.cuda.synchronize()
    return rev


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water", 0])
def test_reverse_slots_exact(key):
    x = _inputs(key)
    rev = _reverse_gpu(x).cpu().numpy()
    assert np.array_equal(rev, _reverse_expected(x.nlist, x.atype, x.cfg.sel))
    # symmetric lists: every valid slot has its reverse
    assert np.all(rev[x.nlist >= 0] >= 0)


def test_reverse_slots_unsorted_lists():
    # shuffled slots inside each sel block: the scan finds the same slots
    x = _inputs("tiny_alloy")
    off = np.concatenate([[0], np.cumsum(x.cfg.sel)])
    rng = np.random.default_rng(3)
    nl = x.nlist.copy()
    for i in range(len(nl)):
        for t in range(x.cfg.ntypes):
            nl[i, off[t]:off[t + 1]] = rng.permutation(nl[i, off[t]:off[t + 1]])
    y = type(x)(**{**x.__dict__, "nlist": nl})
    rev = _reverse_gpu(y).cpu().numpy()
    assert np.array_equal(rev, _reverse_expected(nl, x.atype, x.cfg.sel))


def _force_gpu(x, lam, dtype="f64"):
    import paper_2107_02103_amd as P
    c = x.cfg
    mode = {"f64": P.DPC_F64, "f32": P.DPC_F32}[dtype]
    coord, at, nl = _dev(x)
    rev = _reverse_gpu(x)
    dem = torch.from_numpy(lam.astype(np.float64 if dtype == "f64" else np.float32)).cuda()
    F = torch.full((len(x.atype), 3), float("nan"), dtype=torch.float64, device="cuda")
    V = torch.full((len(x.atype), 9), float("nan"), dtype=torch.float64, device="cuda")
    _, sigma, sigma_all = _stats(x)
    P.dpc_force_a(torch.cuda.current_stream(), mode, len(x.atype), c.ntypes, c.nnei, c.box, c.rc,
                  c.rcs, sigma, sigma_all, coord, at, nl, rev, dem, F, V)
    torch.cuda.synchronize()
    return F.cpu().numpy(), V.cpu().numpy().reshape(-1, 3, 3)


def _lam(x, seed):
    rng = np.random.default_rng([2107_02103, 88, seed])
    return random_grad(rng, len(x.atype), x.cfg.nnei) * (x.nlist >= 0)[..., None]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water", 0])
def test_force_virial_parity(key):
    x = _inputs(key)
    c = x.cfg
    lam = _lam(x, 1)
    F, V = _force_gpu(x, lam)
    Fr, Vr = ev.force_virial(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, *_stats(x), lam)
    ef, evv = _normwise(F, Fr), _normwise(V, Vr)
    print(f"[gpu-env] {c.name} force normwise {ef:.2e} virial {evv:.2e}", flush=True)
    assert ef <= 1e-11 and evv <= 1e-11
    # float32 dE/dR~: the oracle on the rounded input
    F32, V32 = _force_gpu(x, lam, "f32")
    Fr32, Vr32 = ev.force_virial(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, *_stats(x),
                                 lam.astype(np.float32).astype(np.float64))
    assert _normwise(F32, Fr32) <= 1e-11 and _normwise(V32, Vr32) <= 1e-11


@pytest.mark.timeout(600)
@pytest.mark.parametrize("key", [1, 2])
def test_force_properties_at_size(key):
    # forces sum to zero, bitwise reproducible
    x = _inputs(key)
    lam = _lam(x, 2)
    F, V = _force_gpu(x, lam)
    F2, V2 = _force_gpu(x, lam)
    assert np.array_equal(F, F2) and np.array_equal(V, V2)
    tot = np.abs(F.sum(0)).max()
    print(f"[gpu-env] {x.cfg.name} |sum F| {tot:.2e}, max |F| {np.abs(F).max():.2e}", flush=True)
    assert tot <= 1e-10 * np.abs(F).max() * np.sqrt(len(F))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("key", ["tiny_water", "tiny_alloy", 0])
def test_chain_positions_to_forces(key):
    # GPU: env matrix -> forward -> descriptor backward -> backward -> forces,
    # against the oracle's same chain (float64)
    import paper_2107_02103_amd as P
    from oracle.se_a import backward, descriptor_backward, forward
    from oracle.table import build_tables
    x = _inputs(key)
    c = x.cfg
    mean, sigma, sigma_all = _stats(x)
    n = len(x.atype)
    W = random_grad(np.random.default_rng([2107_02103, 99, 1]), n, c.m1, width=c.m2)
    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, c.d1, c.d2, c.sel, c.m2)
    coord, at, nl = _dev(x)
    em = torch.empty((n, c.nnei, 4), dtype=torch.float64, device="cuda")
    P.dpc_env_mat_a(torch.cuda.current_stream(), P.DPC_F64, n, c.ntypes, c.nnei, c.box, c.rc, c.rcs,
                    mean, sigma, sigma_all, coord, at, nl, em)
    T, D = op.forward(em, nl, at)
    dT = op.descriptor_backward(T, torch.from_numpy(W).cuda())
    dR = op.backward(em, nl, at, dT)
    rev = _reverse_gpu(x)
    F = torch.empty((n, 3), dtype=torch.float64, device="cuda")
    P.dpc_force_a(torch.cuda.current_stream(), P.DPC_F64, n, c.ntypes, c.nnei, c.box, c.rc, c.rcs,
                  sigma, sigma_all, coord, at, nl, rev, dR, F, None)
    torch.cuda.synchronize()
    tabs = build_tables(x)
    emr = ev.env_mat(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, mean, sigma, sigma_all)
    Tr, _ = forward(emr, x.nlist, x.atype, tabs, c.sel, c.m2)
    dRr = backward(emr, x.nlist, x.atype, tabs, c.sel, descriptor_backward(Tr, W))
    Fr, _ = ev.force_virial(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, mean, sigma, sigma_all, dRr)
    err = _normwise(F.cpu().numpy(), Fr)
    print(f"[gpu-env] {c.name} chain forces normwise {err:.2e}", flush=True)
    assert err <= 1e-10


@pytest.mark.parametrize("key", ["tiny_water", "tiny_alloy", "cu256"])
def test_chain_energies_and_forces(key):
    # GPU: env matrix -> forward -> fitting net -> descriptor backward ->
    # backward -> forces, against the oracle's same chain (float64)
    import paper_2107_02103_amd as P
    import oracle.fitting as fn
    from oracle.se_a import backward, descriptor_backward, forward
    from oracle.table import build_tables
    from synth.system import random_fitting_net
    x = _inputs(key)
    c = x.cfg
    mean, sigma, sigma_all = _stats(x)
    n = len(x.atype)
    net = random_fitting_net(np.random.default_rng([2107_02103, 99, 2]), c.m1 * c.m2, (240,) * 3)
    keep = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in net["W"] + net["b"] + [net["w_out"]]]
    fnet = P.dpc_fitting_net()
    fnet.n_in, fnet.width, fnet.b_out = c.m1 * c.m2, 240, net["b_out"]
    for l in range(3):
        fnet.W[l] = keep[l].data_ptr()
        fnet.b[l] = keep[3 + l].data_ptr()
    fnet.w_out = keep[6].data_ptr()
    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, c.d1, c.d2, c.sel, c.m2)
    coord, at, nl = _dev(x)
    s = torch.cuda.current_stream()
    em = torch.empty((n, c.nnei, 4), dtype=torch.float64, device="cuda")
    P.dpc_env_mat_a(s, P.DPC_F64, n, c.ntypes, c.nnei, c.box, c.rc, c.rcs, mean, sigma, sigma_all,
                    coord, at, nl, em)
    T, D = op.forward(em, nl, at)
    nb = P.dpc_fitting_workspace_bytes(n, 240)
    ws = torch.empty(nb // 8, dtype=torch.float64, device="cuda")
    E = torch.empty(n, dtype=torch.float64, device="cuda")
    dD = torch.empty_like(D)
    h = P.RocblasHandle()
    P.dpc_fitting_fwd_bwd(s, h.value, n, fnet, D, ws, nb, E, dD)
    dR = op.backward(em, nl, at, op.descriptor_backward(T, dD))
    F = torch.empty((n, 3), dtype=torch.float64, device="cuda")
    P.dpc_force_a(s, P.DPC_F64, n, c.ntypes, c.nnei, c.box, c.rc, c.rcs, sigma, sigma_all, coord, at, nl,
                  _reverse_gpu(x), dR, F, None)
    torch.cuda.synchronize()
    h.close()
    tabs = build_tables(x)
    emr = ev.env_mat(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, mean, sigma, sigma_all)
    Tr, Dr = forward(emr, x.nlist, x.atype, tabs, c.sel, c.m2)
    Er, _ = fn.forward(Dr, net)
    dRr = backward(emr, x.nlist, x.atype, tabs, c.sel, descriptor_backward(Tr, fn.backward(Dr, net)))
    Fr, _ = ev.force_virial(x.coords, c.box, x.atype, x.nlist, c.rc, c.rcs, mean, sigma, sigma_all, dRr)
    eE = np.max(np.abs(E.cpu().numpy() - Er)) / np.max(np.abs(Er))
    eF = _normwise(F.cpu().numpy(), Fr)
    print(f"[gpu-env] {c.name} chain with fitting net: E {eE:.2e} forces normwise {eF:.2e}", flush=True)
    assert eE <= 1e-12 and eF <= 1e-10
