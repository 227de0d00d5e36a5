"""GPU parity of the fitting net (energy and dE/dD) through the C ABI against
the oracle, on a seeded random net and seeded descriptors."""
import numpy as np
import pytest

import oracle.fitting as fn
from synth.system import random_fitting_net, random_grad

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run(n, m1, m2, width, seed, sample=None, device_mode=False):
    import paper_2107_02103_amd as P
    rng = np.random.default_rng([2107_02103, 66, seed])
    net = random_fitting_net(rng, m1 * m2, (width,) * 3)
    D = random_grad(rng, n, m1, width=m2)
    dev = {k: [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in net[k]] for k in ("W", "b")}
    wout = torch.from_numpy(net["w_out"]).cuda()
    c = P.dpc_fitting_net()
    c.n_in, c.width, c.b_out = m1 * m2, width, net["b_out"]
    for l in range(3):
        c.W[l] = dev["W"][l].data_ptr()
        c.b[l] = dev["b"][l].data_ptr()
    c.w_out = wout.data_ptr()
    Dg = torch.from_numpy(D).cuda()
    nb = P.dpc_fitting_workspace_bytes(n, width)
    ws = torch.empty(max(nb, 8) // 8, dtype=torch.float64, device="cuda")
    E = torch.full((n,), float("nan"), dtype=torch.float64, device="cuda")
    G = torch.full((n, m1, m2), float("nan"), dtype=torch.float64, device="cuda")
    h = P.RocblasHandle()
    if device_mode:
        h.set_pointer_mode(1)
    P.dpc_fitting_fwd_bwd(torch.cuda.current_stream(), h.value, n, c, Dg, ws, nb, E, G)
    torch.cuda.synchronize()
    assert h.pointer_mode() == (1 if device_mode else 0)   # the caller's mode is restored
    h.close()
    atoms = np.arange(n) if sample is None else sample
    Er, _ = fn.forward(D[atoms], net)
    Gr = fn.backward(D[atoms], net)
    idx = torch.from_numpy(np.asarray(atoms, np.int64)).cuda()
    E, G = E[idx].cpu().numpy(), G[idx].cpu().numpy()
    eE = np.max(np.abs(E - Er)) / np.max(np.abs(Er))
    eG = max(np.max(np.abs(G[a] - Gr[a])) / np.max(np.abs(Gr[a])) for a in range(len(atoms)))
    print(f"[gpu-fitting] n={n} in={m1 * m2} width={width} atoms={len(atoms)} E {eE:.2e} dE/dD {eG:.2e}",
          flush=True)
    return eE, eG


@pytest.mark.parametrize("n,m1,m2,width", [(37, 100, 16, 240), (5, 3, 2, 7), (1, 1, 1, 1), (300, 20, 4, 33)])
def test_parity(n, m1, m2, width):
    eE, eG = _run(n, m1, m2, width, seed=n + width)
    assert eE <= 1e-12 and eG <= 1e-12


def test_caller_handle_in_device_pointer_mode():
    # the entry point passes alpha and beta from the host whatever the
    # handle's mode, and gives the handle back in the caller's mode
    eE, eG = _run(19, 10, 4, 24, seed=5, device_mode=True)
    assert eE <= 1e-12 and eG <= 1e-12


@pytest.mark.timeout(600)
def test_parity_full_size_cu1m_sampled():
    n = 1 << 20
    sample = np.unique(np.concatenate([np.random.default_rng(3).choice(n, 48, replace=False), [0, n - 1]]))
    eE, eG = _run(n, 100, 16, 240, seed=7, sample=sample)
    assert eE <= 1e-12 and eG <= 1e-12


def test_saturated_and_nan_inputs():
    # descriptors scaled by 50 drive |z| far past 20 (tanh rounds to +-1
    # there); a NaN descriptor stays in its own atom's energy and gradient
    import paper_2107_02103_amd as P
    n, m1, m2, width = 9, 10, 4, 24
    rng = np.random.default_rng([2107_02103, 66, 99])
    net = random_fitting_net(rng, m1 * m2, (width,) * 3)
    D = 50.0 * random_grad(rng, n, m1, width=m2)
    D[4, 3, 1] = np.nan
    dev = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in net["W"] + net["b"] + [net["w_out"]]]
    c = P.dpc_fitting_net()
    c.n_in, c.width, c.b_out = m1 * m2, width, net["b_out"]
    for l in range(3):
        c.W[l] = dev[l].data_ptr()
        c.b[l] = dev[3 + l].data_ptr()
    c.w_out = dev[6].data_ptr()
    nb = P.dpc_fitting_workspace_bytes(n, width)
    ws = torch.empty(nb // 8, dtype=torch.float64, device="cuda")
    E = torch.empty(n, dtype=torch.float64, device="cuda")
    G = torch.empty((n, m1, m2), dtype=torch.float64, device="cuda")
    h = P.RocblasHandle()
    P.dpc_fitting_fwd_bwd(torch.cuda.current_stream(), h.value, n, c, torch.from_numpy(D).cuda(), ws, nb, E, G)
    torch.cuda.synchronize()
    h.close()
    E, G = E.cpu().numpy(), G.cpu().numpy()
    ok = np.arange(n) != 4
    assert np.isnan(E[4]) and np.all(np.isnan(G[4]))
    Er, _ = fn.forward(D[ok], net)
    Gr = fn.backward(D[ok], net)
    eE = np.max(np.abs(E[ok] - Er)) / np.max(np.abs(Er))
    eG = max(np.max(np.abs(G[ok][a] - Gr[a])) / max(np.max(np.abs(Gr[a])), 1e-300) for a in range(len(Gr)))
    print(f"[gpu-fitting] saturated inputs: E {eE:.2e} dE/dD {eG:.2e}", flush=True)
    assert eE <= 1e-12 and eG <= 1e-12
