"""The backward from dE/dD (dpc_se_a_tab_bwd_from_dD: the descriptor backward
fused into the matrix-core backward) against the oracle chain
descriptor_backward -> backward, and against the two separate GPU calls.
Inputs: the workloads' R~, neighbour lists and tables, with seeded
standard-normal T and dE/dD (any T, dE/dD is a valid input)."""
import numpy as np
import pytest

from synth import make_inputs
from synth.configs import get_config
from synth.system import random_grad

from parity import normwise

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-12


def _oracle(x, T, dD, atoms):
    from oracle import cref
    from oracle.se_a import descriptor_backward
    from oracle.table import build_tables
    dT = descriptor_backward(T[atoms], dD[atoms])
    pb = cref.Problem(x.em[atoms], x.nlist[atoms], x.atype[atoms], build_tables(x), x.cfg.sel, x.cfg.m2)
    return pb.backward(dT)


def _gpu(x, T, dD):
    import paper_2107_02103_amd as P
    c = x.cfg
    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, c.d1, c.d2, c.sel, c.m2)
    em = torch.from_numpy(x.em).cuda()
    nl = torch.from_numpy(x.nlist).cuda()
    at = torch.from_numpy(x.atype).cuda()
    Tg = torch.from_numpy(T).cuda()
    Dg = torch.from_numpy(dD).cuda()
    fused = op.backward_from_dD(em, nl, at, Tg, Dg)
    two = op.backward(em, nl, at, op.descriptor_backward(Tg, Dg))
    torch.cuda.synchronize()
    return fused.cpu().numpy(), two.cpu().numpy()


def _grads(x, seed):
    rng = np.random.default_rng([2107_02103, 55, seed])
    n, c = x.nlist.shape[0], x.cfg
    return random_grad(rng, n, c.m1), random_grad(rng, n, c.m1, width=c.m2)


@pytest.mark.parametrize("key", ["tiny_fcc", "tiny_alloy", "tiny_water", 0, 1, 2])
def test_fused_matches_oracle_chain(key):
    x = make_inputs(get_config(key), with_grad=False)
    T, dD = _grads(x, 1)
    fused, two = _gpu(x, T, dD)
    n = len(x.atype)
    atoms = np.unique(np.concatenate([np.random.default_rng(0).choice(n, min(n, 200), replace=False),
                                      [0, n - 1]]))
    ref = _oracle(x, T, dD, atoms)
    e_oracle, e_two = normwise(fused[atoms], ref), normwise(fused, two)
    print(f"[fused-bwd] {x.cfg.name}: vs oracle {e_oracle:.2e} ({len(atoms)} atoms), "
          f"vs two calls {e_two:.2e} (all {n})", flush=True)
    assert e_oracle <= TOL and e_two <= TOL
    assert np.all(fused[x.nlist < 0] == 0)


@pytest.mark.timeout(600)
def test_fused_full_size_cu1m():
    x = make_inputs(get_config(3), with_grad=False)
    T, dD = _grads(x, 3)
    fused, two = _gpu(x, T, dD)
    atoms = np.unique(np.concatenate([np.random.default_rng(3).choice(len(fused), 40, replace=False),
                                      [0, len(fused) - 1]]))
    e_oracle = normwise(fused[atoms], _oracle(x, T, dD, atoms))
    e_two = max(normwise(fused[a:a + 65536], two[a:a + 65536]) for a in range(0, len(fused), 65536))
    print(f"[fused-bwd] cu1m: vs oracle {e_oracle:.2e}, vs two calls {e_two:.2e} (all atoms)", flush=True)
    assert e_oracle <= TOL and e_two <= TOL


@pytest.mark.parametrize("sel,m1,m2", [((77,), 17, 4), ((3, 70), 100, 16), ((40, 33), 128, 16),
                                       ((20,), 113, 2), ((700, 900), 100, 16), ((64,), 64, 8)])
def test_fused_edge_shapes(sel, m1, m2):
    from synth.edge import edge_inputs
    x = edge_inputs(37, sel, m1, m2, seed=sum(sel) + m1 + 11)
    x.nlist[5] = -1
    x.em[5] = 0
    T, dD = _grads(x, m1)
    T[9, :, :] = 0.0                      # an atom with zero T: zero dE/dT
    fused, two = _gpu(x, T, dD)
    atoms = np.arange(37)
    assert normwise(fused, _oracle(x, T, dD, atoms)) <= TOL
    assert normwise(fused, two) <= TOL
    assert np.all(fused[5] == 0)


def test_fused_refuses_unsupported_shapes_and_nan_stays():
    import paper_2107_02103_amd as P
    from synth.edge import edge_inputs
    x = edge_inputs(9, (50,), 100, 16, seed=4)
    T, dD = _grads(x, 2)
    dD[3, 7, 5] = np.nan
    fused, _ = _gpu(x, T, dD)
    others = [i for i in range(9) if i != 3]
    assert np.isnan(fused[3]).any() and np.isfinite(fused[others]).all()
    assert normwise(fused[others], _oracle(x, T, dD, np.array(others))) <= TOL
    for m1, m2, dt in ((100, 15, P.DPC_F64), (129, 16, P.DPC_F64), (100, 32, P.DPC_F64),
                       (100, 16, P.DPC_F32)):
        with pytest.raises(P.DpcError) as e:
            P.dpc_se_a_tab_bwd_from_dD(0, dt, 4, 1, [8], m1, m2,
                                       P.make_ranges([0.0], [0.01], [10], [0.1], [1]),
                                       4096, 4096, 4096, 4096, 4096, 4096, 4096)
        assert e.value.status == P.DPC_ENOTSUP, (m1, m2, dt)
