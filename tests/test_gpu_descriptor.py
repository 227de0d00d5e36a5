"""GPU parity of the descriptor backward (dE/dT from dE/dD and T) through the
C ABI against the oracle, on seeded synthetic T and dE/dD (standard normal,
the shapes of the five workloads' descriptors: M = 100, M' = 16, and edge
shapes)."""
import numpy as np
import pytest

from oracle.se_a import descriptor_backward
from synth.system import random_grad

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _inputs(nat, m1, m2, seed):
    rng = np.random.default_rng([2107_02103, 77, seed])
    return random_grad(rng, nat, m1), random_grad(rng, nat, m1, width=m2)


def _gpu(T, dD, dtype):
    import paper_2107_02103_amd as P
    mode = {"f64": P.DPC_F64, "f32": P.DPC_F32, "f32acc64": P.DPC_F32_ACC64}[dtype]
    t_in = np.float32 if dtype == "f32" else np.float64
    t_out = torch.float64 if dtype == "f64" else torch.float32
    Tg = torch.from_numpy(T.astype(t_in)).cuda()
    Dg = torch.from_numpy(dD.astype(t_in)).cuda()
    out = torch.full(T.shape, float("nan"), dtype=t_out, device="cuda")
    P.dpc_descriptor_bwd(torch.cuda.current_stream(), mode, T.shape[0], T.shape[1], dD.shape[2],
                         Tg, Dg, out)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def _check(T, dD, got, dtype, atoms):
    # the oracle on the inputs as the kernel saw them (float32-rounded for f32)
    if dtype == "f32":
        T = T.astype(np.float32).astype(np.float64)
        dD = dD.astype(np.float32).astype(np.float64)
    ref = descriptor_backward(T[atoms], dD[atoms])
    g = got[atoms]
    # bound of the terms' magnitudes: the same sums over absolute values
    m2 = dD.shape[2]
    aT, aD = np.abs(T[atoms]), np.abs(dD[atoms])
    A = aD @ aT[:, :m2, :]
    A[:, :m2, :] += np.transpose(aD, (0, 2, 1)) @ aT
    tol = {"f64": 1e-12, "f32": 1e-5, "f32acc64": 1e-6}[dtype]
    comp = np.max(np.abs(g - ref) / (A + 1e-300))
    norm = max(np.max(np.abs(g[a] - ref[a])) / np.max(np.abs(ref[a])) for a in range(len(atoms)))
    print(f"[gpu-descriptor] {dtype} atoms={len(atoms)} M={T.shape[1]} M'={m2} "
          f"componentwise {comp:.2e} normwise {norm:.2e}", flush=True)
    assert comp <= tol and norm <= tol


@pytest.mark.parametrize("dtype", ["f64", "f32", "f32acc64"])
def test_parity_workload_shape(dtype):
    # 37 atoms: several workgroups and a ragged last one
    T, dD = _inputs(37, 100, 16, seed=1)
    got = _gpu(T, dD, dtype)
    _check(T, dD, got, dtype, np.arange(37))


@pytest.mark.parametrize("m1,m2", [(1, 1), (17, 4), (64, 64), (129, 8), (256, 16), (100, 1),
                                   (5, 5), (16, 16), (37, 16), (128, 16)])
def test_parity_edge_shapes(m1, m2):
    T, dD = _inputs(9, m1, m2, seed=m1 * 7 + m2)
    _check(T, dD, _gpu(T, dD, "f64"), "f64", np.arange(9))


@pytest.mark.parametrize("dtype", ["f64", "f32acc64"])
def test_parity_several_atoms_per_wavefront(dtype):
    # more atoms than wavefronts in the grid of the M' = 16 kernel, ragged
    T, dD = _inputs(5003, 100, 16, seed=21)
    got = _gpu(T, dD, dtype)
    atoms = np.unique(np.concatenate([np.random.default_rng(2).choice(5003, 60, replace=False),
                                      [0, 1, 4095, 4096, 5002]]))
    _check(T, dD, got, dtype, atoms)


def test_unaligned_buffers_take_the_general_kernel():
    import paper_2107_02103_amd as P
    T, dD = _inputs(7, 100, 16, seed=5)
    # views 8 bytes into flat buffers: not 16-byte aligned
    bt = torch.zeros(T.size + 1, dtype=torch.float64, device="cuda")
    bd = torch.zeros(dD.size + 1, dtype=torch.float64, device="cuda")
    bo = torch.full((T.size + 1,), float("nan"), dtype=torch.float64, device="cuda")
    bt[1:] = torch.from_numpy(T.ravel()).cuda()
    bd[1:] = torch.from_numpy(dD.ravel()).cuda()
    P.dpc_descriptor_bwd(torch.cuda.current_stream(), P.DPC_F64, 7, 100, 16, bt.data_ptr() + 8,
                         bd.data_ptr() + 8, bo.data_ptr() + 8)
    torch.cuda.synchronize()
    got = bo[1:].cpu().numpy().reshape(T.shape)
    _check(T, dD, got, "f64", np.arange(7))


def test_too_large_for_lds_is_refused():
    import paper_2107_02103_amd as P
    T = torch.zeros((2, 100, 4), dtype=torch.float64, device="cuda")
    dD = torch.zeros((2, 100, 100), dtype=torch.float64, device="cuda")
    out = torch.zeros_like(T)
    with pytest.raises(P.DpcError) as e:
        P.dpc_descriptor_bwd(0, P.DPC_F64, 2, 100, 100, T, dD, out)
    assert e.value.status == P.DPC_ENOTSUP


@pytest.mark.timeout(600)
def test_parity_full_size_cu1m_sampled():
    # the cu1m descriptor (1,048,576 atoms, M = 100, M' = 16) in the launch
    # configuration bench.py times; sampled atoms against the oracle
    n = 1 << 20
    print("[gpu-descriptor] generating cu1m-shaped T and dE/dD", flush=True)
    T, dD = _inputs(n, 100, 16, seed=3)
    got = _gpu(T, dD, "f64")
    rng = np.random.default_rng(11)
    atoms = np.unique(np.concatenate([rng.choice(n, 40, replace=False), [0, n - 1]]))
    _check(T, dD, got, "f64", atoms)
    assert np.isfinite(got).all()
