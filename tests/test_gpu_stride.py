"""Table-stride study (the paper varies the tabulation stride, Sec. III): the
GPU kernels with tables of stride 0.1, 0.01 and 0.001 (band stride 10x)
against the original, un-tabulated embedding net (the oracle's
forward_untabulated / backward_untabulated) on sampled atoms of the
water4096 and alcumg32000 workloads.  The error must fall with the stride as
the quintic Hermite remainder (order 6) until rounding takes over."""
import numpy as np
import pytest

from oracle.se_a import backward_untabulated, forward_untabulated
from synth import make_inputs
from synth.configs import get_config

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

_CACHE = {}


def _inputs(key, d1):
    k = (key, d1)
    if k not in _CACHE:
        print(f"[gpu-stride] generating {key} stride {d1}", flush=True)
        _CACHE[k] = make_inputs(get_config(key).with_(d1=d1, d2=10 * d1))
    return _CACHE[k]


def _errors(key, d1, dtype, atoms_n=24):
    import paper_2107_02103_amd as P
    x = _inputs(key, d1)
    c = x.cfg
    mode = {"f64": P.DPC_F64, "f32": P.DPC_F32}[dtype]
    store = np.float64 if dtype == "f64" else np.float32
    op = P.SeATab(x.nets, x.lo, x.L1, x.L2, c.d1, c.d2, c.sel, c.m2, dtype=mode)
    em = torch.from_numpy(x.em.astype(store)).cuda()
    nl = torch.from_numpy(x.nlist).cuda()
    at = torch.from_numpy(x.atype).cuda()
    dT = torch.from_numpy(x.dT.astype(store)).cuda()
    T, D = op.forward(em, nl, at)
    dR = op.backward(em, nl, at, dT)
    torch.cuda.synchronize()
    n = x.nlist.shape[0]
    atoms = np.unique(np.concatenate([np.random.default_rng(4).choice(n, atoms_n, replace=False), [0]]))
    em64 = x.em.astype(store).astype(np.float64)
    dT64 = x.dT.astype(store).astype(np.float64)
    Tu, Du = forward_untabulated(em64, x.nlist, x.atype, x.nets, c.sel, c.m2, atoms=atoms)
    dRu = backward_untabulated(em64, x.nlist, x.atype, x.nets, c.sel, dT64, atoms=atoms)
    out = {}
    for name, g, r in (("T", T, Tu), ("D", D, Du), ("dR", dR, dRu)):
        g = g.cpu().numpy()[atoms].astype(np.float64)
        out[name] = max(np.max(np.abs(g[a] - r[a])) / np.max(np.abs(r[a])) for a in range(len(atoms)))
    mb = op.coeff.numel() * op.coeff.element_size() / 1e6
    print(f"[gpu-stride] {key} {dtype} stride {d1}: intervals {int(x.L1.max())}+{int(x.L2.max())} "
          f"per pair, table {mb:.2f} MB, normwise error vs the net T {out['T']:.2e} "
          f"D {out['D']:.2e} dE/dR {out['dR']:.2e}", flush=True)
    return out


@pytest.mark.timeout(600)
@pytest.mark.parametrize("key", ["water4096", "alcumg32000"])
def test_error_falls_with_stride(key):
    e = {d1: _errors(key, d1, "f64") for d1 in (0.1, 0.01, 0.001)}
    # the paper's working stride: tabulation error far below the model error
    assert e[0.01]["T"] <= 1e-9 and e[0.01]["D"] <= 1e-9 and e[0.01]["dR"] <= 1e-7
    # the remainder is of order 6 in the stride for g (T, D) and of order 5
    # for g' (dE/dR~): 10x finer, 10^6 and 10^5 smaller, until rounding takes
    # over -- for g' at a floor near eps / stride, since the table's highest
    # coefficients carry rounding of order eps / stride^k against t^k
    for q in ("T", "D"):
        assert e[0.01][q] <= max(e[0.1][q] * 1e-4, 1e-13)
        assert e[0.001][q] <= max(e[0.01][q] * 1e-3, 1e-13)
    assert e[0.01]["dR"] <= max(e[0.1]["dR"] * 1e-3, 1e-14 / 0.01)
    assert e[0.001]["dR"] <= max(e[0.01]["dR"] * 1e-2, 1e-14 / 0.001)


@pytest.mark.timeout(600)
def test_float32_error_is_rounding_not_tabulation():
    e = _errors("water4096", 0.01, "f32")
    assert max(e.values()) <= 1e-4
