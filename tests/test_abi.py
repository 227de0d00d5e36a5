"""C-ABI checks that need no GPU: exported symbols, table layout, the host
table builder against the oracle (by evaluation) and argument validation."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_2107_02103_amd as P
from paper_2107_02103_amd import binding as B
from oracle.table import build_table as oracle_table
from synth import make_inputs
from synth.configs import get_config
from synth.system import random_net

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dpc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dpc_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = _declared()
    assert set(names) == set(B.EXPORTED)
    lib = C.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_strerror_and_version():
    assert P.dpc_version() >= 100
    for s in (0, -1, -2, -3, -4, -5):
        assert len(P.dpc_strerror(s)) > 1
    assert P.dpc_strerror(-99) == "unknown status"


def test_table_layout_offsets():
    r = P.make_ranges([0.0, -1.0], [0.01, 0.02], [10, 20], [0.1, 0.1], [2, 3], )
    nbytes = P.dpc_table_layout(r, 7, P.DPC_F64)
    assert r[0].offset == 0 and r[1].offset == 12 * 6 * 8        # rows padded to 8 channels
    assert nbytes == (12 + 23) * 6 * 8 * 8
    assert P.dpc_table_layout(r, 7, P.DPC_F32) == nbytes // 2


@pytest.mark.parametrize("bad,code", [
    (dict(d1=0.0), B.DPC_ERANGE), (dict(d2=-0.1), B.DPC_ERANGE), (dict(L1=0), B.DPC_ERANGE),
    (dict(L2=0), B.DPC_ERANGE), (dict(lo=float("nan")), B.DPC_ERANGE)])
def test_table_layout_rejects_bad_ranges(bad, code):
    kw = dict(lo=0.0, d1=0.01, L1=5, d2=0.1, L2=1)
    kw.update(bad)
    r = P.make_ranges([kw["lo"]], [kw["d1"]], [kw["L1"]], [kw["d2"]], [kw["L2"]])
    with pytest.raises(P.DpcError) as e:
        P.dpc_table_layout(r, 4, P.DPC_F64)
    assert e.value.status == code


def test_table_layout_rejects_bad_sizes():
    r = P.make_ranges([0.0], [0.01], [5], [0.1], [1])
    for m1, dt, code in ((0, 0, B.DPC_EINVAL), (257, 0, B.DPC_ENOTSUP), (4, 7, B.DPC_EINVAL)):
        with pytest.raises(P.DpcError) as e:
            P.dpc_table_layout(r, m1, dt)
        assert e.value.status == code


def _eval_lib(buf, rng, m1, x):
    """Value/slope/curvature of the library's table at x (test-side Horner)."""
    L1, L2 = rng.L1, rng.L2
    ld = B.table_ld(m1)
    c = B.unpack_table(buf[rng.offset:rng.offset + (L1 + L2) * 6 * ld], L1 + L2, ld)[:, :, :m1]
    c = c.astype(np.float64)
    x_up = rng.lo + L1 * rng.d1
    l = np.where(x < x_up, np.clip(np.floor((x - rng.lo) / rng.d1), 0, L1 - 1),
                 L1 + np.clip(np.floor((x - x_up) / rng.d2), 0, L2 - 1)).astype(int)
    t = np.where(l < L1, x - (rng.lo + l * rng.d1), x - (x_up + (l - L1) * rng.d2))[:, None]
    q = c[l]                                      # [n, 6, m1]
    g = sum(q[:, k] * t ** k for k in range(6))
    g1 = sum(k * q[:, k] * t ** (k - 1) for k in range(1, 6))
    g2 = sum(k * (k - 1) * q[:, k] * t ** (k - 2) for k in range(2, 6))
    return g, g1, g2


@pytest.mark.parametrize("seed,widths", [(0, (1, 25, 50, 100)), (1, (1, 4, 8, 16)), (2, (1, 3, 6, 6))])
def test_build_table_matches_oracle_by_evaluation(seed, widths):
    net = random_net(np.random.default_rng(seed), widths)
    lo, d1, L1, d2, L2 = -0.7, 0.01, 450, 0.1, 45
    r = P.make_ranges([lo], [d1], [L1], [d2], [L2])
    buf = P.build_tables([net], r, P.DPC_F64)
    ot = oracle_table(net, lo, d1, L1, d2, L2)
    x = np.random.default_rng(seed).uniform(lo, ot.x_end - 1e-9, 5000)
    g, g1, g2 = _eval_lib(buf, r[0], widths[-1], x)
    o, o1, o2 = ot.evaluate(x, order=2)
    s = np.max(np.abs(o))
    assert np.max(np.abs(g - o)) <= 1e-13 * s
    assert np.max(np.abs(g1 - o1)) <= 1e-9 * np.max(np.abs(o1))
    assert np.max(np.abs(g2 - o2)) <= 1e-5 * np.max(np.abs(o2))


def test_table_padding_is_zero():
    net = random_net(np.random.default_rng(4), (1, 3, 6, 6))    # m1 = 6 -> rows of 8
    r = P.make_ranges([-0.5], [0.01], [20], [0.1], [2])
    buf = B.unpack_table(P.build_tables([net], r, P.DPC_F64), 22, 8)
    assert np.all(buf[:, :, 6:] == 0) and np.any(buf[:, :, :6] != 0)


def test_build_table_f32_is_rounded_f64():
    net = random_net(np.random.default_rng(3), (1, 25, 50, 100))
    r = P.make_ranges([-0.5], [0.01], [100], [0.1], [10])
    b64 = P.build_tables([net], r, P.DPC_F64)
    r32 = P.make_ranges([-0.5], [0.01], [100], [0.1], [10])
    b32 = P.build_tables([net], r32, P.DPC_F32)
    np.testing.assert_array_equal(b32, b64.astype(np.float32))


def test_build_table_rejects_bad_nets():
    net = random_net(np.random.default_rng(3), (1, 4, 8))
    r = P.make_ranges([-0.5], [0.01], [10], [0.1], [1])
    out = np.zeros((11 * 6 * 8,))
    bad = {"W": [np.zeros((2, 4)), net["W"][1]], "b": net["b"]}     # widths[0] != 1
    with pytest.raises(P.DpcError) as e:
        P.dpc_build_table(bad, r[0], P.DPC_F64, out)
    assert e.value.status == B.DPC_EINVAL
    with pytest.raises(ValueError):                                   # output too small
        P.dpc_build_table(net, r[0], P.DPC_F64, np.zeros(10))


def test_kernel_entry_points_validate_before_launch():
    # every call below must fail (or no-op) on the host without touching HIP
    sel = [4, 4]
    r = P.make_ranges([0.0] * 4, [0.01] * 4, [5] * 4, [0.1] * 4, [1] * 4)
    P.dpc_table_layout(r, 8, P.DPC_F64)
    fake = 4096  # never dereferenced: validation fails first
    cases = [
        (dict(dtype=9), B.DPC_EINVAL), (dict(m2=9), B.DPC_EINVAL), (dict(m2=0), B.DPC_EINVAL),
        (dict(ntypes=9, sel=[1] * 9), B.DPC_ENOTSUP), (dict(m1=300, m2=4), B.DPC_ENOTSUP),
        (dict(nloc=-1), B.DPC_EINVAL), (dict(sel=[4, -1]), B.DPC_EINVAL),
        (dict(em=0), B.DPC_EINVAL), (dict(T=0), B.DPC_EINVAL),
        (dict(em=fake + 8), B.DPC_EINVAL),                         # R~ not 16-byte aligned
    ]
    for kw, code in cases:
        a = dict(stream=0, dtype=P.DPC_F64, nloc=3, ntypes=2, sel=sel, m1=8, m2=4, ranges=r,
                 coeff=fake, atype=fake, nlist=fake, em=fake, T=fake, D=fake)
        a.update(kw)
        if "ntypes" in kw:
            a["ranges"] = P.make_ranges([0.0] * 81, [0.01] * 81, [5] * 81, [0.1] * 81, [1] * 81)
        with pytest.raises(P.DpcError) as e:
            P.dpc_se_a_tab_fwd(**a)
        assert e.value.status == code, kw
    bad = P.make_ranges([0.0] * 4, [0.01] * 4, [5] * 4, [0.0] * 4, [1] * 4)
    with pytest.raises(P.DpcError) as e:
        P.dpc_se_a_tab_bwd(0, P.DPC_F64, 3, 2, sel, 8, bad, fake, fake, fake, fake, fake, fake)
    assert e.value.status == B.DPC_ERANGE
    with pytest.raises(P.DpcError) as e:
        P.dpc_se_a_tab_bwd(0, P.DPC_F64, 3, 2, sel, 8, r, fake, fake, fake, fake + 8, fake, fake)
    assert e.value.status == B.DPC_EINVAL
    with pytest.raises(P.DpcError) as e:                              # dE/dR~ not 16-byte aligned
        P.dpc_se_a_tab_bwd(0, P.DPC_F64, 3, 2, sel, 8, r, fake, fake, fake, fake, fake, fake + 8)
    assert e.value.status == B.DPC_EINVAL
    # nloc = 0 is a no-op that launches nothing
    P.dpc_se_a_tab_fwd(0, P.DPC_F64, 0, 2, sel, 8, 4, r, 0, 0, 0, 0, 0, 0)
    P.dpc_se_a_tab_bwd(0, P.DPC_F64, 0, 2, sel, 8, r, 0, 0, 0, 0, 0, 0)


def test_descriptor_bwd_validates_before_launch():
    fake = 4096  # never dereferenced: validation fails first
    cases = [((9, 3, 8, 4), B.DPC_EINVAL), ((0, -1, 8, 4), B.DPC_EINVAL), ((0, 3, 8, 9), B.DPC_EINVAL),
             ((0, 3, 8, 0), B.DPC_EINVAL), ((0, 3, 0, 1), B.DPC_EINVAL), ((0, 3, 300, 4), B.DPC_ENOTSUP)]
    for (dt, nloc, m1, m2), code in cases:
        with pytest.raises(P.DpcError) as e:
            P.dpc_descriptor_bwd(0, dt, nloc, m1, m2, fake, fake, fake)
        assert e.value.status == code, (dt, nloc, m1, m2)
    for i in range(3):                                                # a null buffer
        ptrs = [fake, fake, fake]
        ptrs[i] = 0
        with pytest.raises(P.DpcError) as e:
            P.dpc_descriptor_bwd(0, P.DPC_F64, 3, 8, 4, *ptrs)
        assert e.value.status == B.DPC_EINVAL
    P.dpc_descriptor_bwd(0, P.DPC_F64, 0, 8, 4, 0, 0, 0)              # nloc = 0: no-op


def test_env_entry_points_validate_before_launch():
    fake = 4096  # never dereferenced: validation fails first
    m = [0.1, 0.2]; sg = [1.0, 1.0]; sa = [1.0, 1.0]
    env = dict(stream=0, dtype=P.DPC_F64, nloc=3, ntypes=2, nnei=8, box=20.0, rc=6.0, rcs=0.5,
               mean=m, sigma=sg, sigma_all=sa, coord=fake, atype=fake, nlist=fake, em=fake)
    cases = [(dict(dtype=7), B.DPC_EINVAL), (dict(nloc=-1), B.DPC_EINVAL), (dict(nnei=0), B.DPC_EINVAL),
             (dict(box=11.0), B.DPC_ERANGE), (dict(rcs=6.0), B.DPC_ERANGE), (dict(rc=-1.0), B.DPC_ERANGE),
             (dict(sigma=[1.0, 0.0]), B.DPC_ERANGE), (dict(sigma_all=[-1.0, 1.0]), B.DPC_ERANGE),
             (dict(ntypes=9, mean=[0.0] * 9, sigma=[1.0] * 9, sigma_all=[1.0] * 9), B.DPC_ENOTSUP),
             (dict(coord=0), B.DPC_EINVAL), (dict(em=0), B.DPC_EINVAL)]
    for kw, code in cases:
        a = dict(env); a.update(kw)
        with pytest.raises(P.DpcError) as e:
            P.dpc_env_mat_a(**a)
        assert e.value.status == code, kw
    f = dict(stream=0, dtype=P.DPC_F64, nloc=3, ntypes=2, nnei=8, box=20.0, rc=6.0, rcs=0.5,
             sigma=sg, sigma_all=sa, coord=fake, atype=fake, nlist=fake, rev=fake, dE_dem=fake,
             force=fake, virial=None)
    for kw, code in [(dict(box=5.0), B.DPC_ERANGE), (dict(rev=0), B.DPC_EINVAL), (dict(force=0), B.DPC_EINVAL),
                     (dict(dtype=5), B.DPC_EINVAL)]:
        a = dict(f); a.update(kw)
        with pytest.raises(P.DpcError) as e:
            P.dpc_force_a(**a)
        assert e.value.status == code, kw
    for kw, code in [(dict(sel=[4, -1]), B.DPC_EINVAL), (dict(box=-1.0), B.DPC_ERANGE),
                     (dict(rev=0), B.DPC_EINVAL)]:
        a = dict(stream=0, nloc=3, ntypes=2, sel=[4, 4], box=20.0, coord=fake, atype=fake, nlist=fake,
                 rev=fake)
        a.update(kw)
        with pytest.raises(P.DpcError) as e:
            P.dpc_nlist_reverse(**a)
        assert e.value.status == code, kw
    # nloc = 0: no-ops
    P.dpc_env_mat_a(**{**env, "nloc": 0, "coord": 0, "em": 0})
    P.dpc_force_a(**{**f, "nloc": 0, "rev": 0, "force": 0})
    P.dpc_nlist_reverse(0, 0, 2, [4, 4], 20.0, 0, 0, 0, 0)


def test_fitting_entry_point_validates_before_launch():
    fake = 4096
    assert P.dpc_fitting_workspace_bytes(10, 240) == 5 * 10 * 240 * 8
    assert P.dpc_fitting_workspace_bytes(5, 7) == 5 * 36 * 8
    assert P.dpc_fitting_workspace_bytes(-1, 240) == 0
    net = P.dpc_fitting_net()
    net.n_in, net.width = 16, 8
    for l in range(3):
        net.W[l] = fake
        net.b[l] = fake
    net.w_out = fake
    nb = P.dpc_fitting_workspace_bytes(4, 8)
    cases = [(dict(nloc=-1), B.DPC_EINVAL), (dict(blas=0), B.DPC_EINVAL), (dict(D=0), B.DPC_EINVAL),
             (dict(workspace_bytes=nb - 8), B.DPC_EINVAL), (dict(workspace=fake + 8), B.DPC_EINVAL),
             (dict(E=0), B.DPC_EINVAL)]
    for kw, code in cases:
        a = dict(stream=0, blas=fake, nloc=4, net=net, D=fake, workspace=fake, workspace_bytes=nb, E=fake,
                 dE_dD=None)
        a.update(kw)
        with pytest.raises(P.DpcError) as e:
            P.dpc_fitting_fwd_bwd(**a)
        assert e.value.status == code, kw
    net.W[1] = 0
    with pytest.raises(P.DpcError) as e:
        P.dpc_fitting_fwd_bwd(0, fake, 4, net, fake, fake, nb, fake)
    assert e.value.status == B.DPC_EINVAL
    net.W[1] = fake
    P.dpc_fitting_fwd_bwd(0, 0, 0, net, 0, 0, 0, 0)                   # nloc = 0: no-op


def test_missing_library_fails_loudly(tmp_path):
    # the product path has no fallback: without the built library the first
    # use of any entry point raises ImportError
    import shutil
    import subprocess
    import sys
    pkg = tmp_path / "paper_2107_02103_amd"
    pkg.mkdir()
    for f in os.listdir(os.path.join(ROOT, "paper_2107_02103_amd")):
        if f.endswith(".py"):                 # the package without its built _lib/
            shutil.copy(os.path.join(ROOT, "paper_2107_02103_amd", f), pkg / f)
    code = "import paper_2107_02103_amd as P; P.dpc_version()"
    r = subprocess.run([sys.executable, "-c", code], cwd=str(tmp_path), capture_output=True, text=True,
                       timeout=300)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "libdpc.so not found" in r.stderr


def test_binding_refuses_undersized_tensors():
    # device buffers carry no size through the C ABI: the binding checks the
    # tensors it is given before the call (CPU tensors suffice here)
    torch = pytest.importorskip("torch")
    f64 = lambda n: torch.zeros(n, dtype=torch.float64)
    i32 = lambda n: torch.zeros(n, dtype=torch.int32)
    with pytest.raises(ValueError, match="dE_dT"):
        P.dpc_descriptor_bwd(0, P.DPC_F64, 3, 8, 4, f64(3 * 8 * 4), f64(3 * 8 * 4), f64(3 * 8 * 4 - 1))
    with pytest.raises(ValueError, match="em"):
        P.dpc_env_mat_a(0, P.DPC_F64, 2, 1, 5, 20.0, 6.0, 0.5, [0.0], [1.0], [1.0], f64(6), i32(2), i32(10),
                        f64(2 * 5 * 4 - 1))
    with pytest.raises(ValueError, match="rev"):
        P.dpc_nlist_reverse(0, 2, 1, [5], 20.0, f64(6), i32(2), i32(10), i32(9))
    with pytest.raises(ValueError, match="virial"):
        P.dpc_force_a(0, P.DPC_F64, 2, 1, 5, 20.0, 6.0, 0.5, [1.0], [1.0], f64(6), i32(2), i32(10), i32(10),
                      f64(40), f64(6), f64(17))
    net = P.dpc_fitting_net()
    net.n_in, net.width = 16, 8
    with pytest.raises(ValueError, match="D"):
        P.dpc_fitting_fwd_bwd(0, 1, 4, net, f64(63), f64(1000), 8000, f64(4))
    with pytest.raises(ValueError, match="workspace"):
        P.dpc_fitting_fwd_bwd(0, 1, 4, net, f64(64), f64(99), 800, f64(4))
    with pytest.raises(ValueError, match="nlist"):
        P.dpc_se_a_tab_fwd(0, P.DPC_F64, 2, 1, [5], 8, 4, None, 0, i32(2), i32(9), f64(40), f64(64), f64(64))


def test_binding_refuses_host_tensors():
    # a correctly sized tensor in host memory would pass its host address to
    # the kernels: the binding refuses it before any call into the library
    torch = pytest.importorskip("torch")
    f64 = lambda n: torch.zeros(n, dtype=torch.float64)
    i32 = lambda n: torch.zeros(n, dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU"):
        P.dpc_descriptor_bwd(0, P.DPC_F64, 3, 8, 4, f64(3 * 8 * 4), f64(3 * 8 * 4), f64(3 * 8 * 4))
    with pytest.raises(ValueError, match="GPU"):
        P.dpc_se_a_tab_fwd(0, P.DPC_F64, 2, 1, [5], 8, 4, None, f64(8), i32(2), i32(10), f64(40),
                           f64(64), f64(64))
    with pytest.raises(ValueError, match="GPU"):
        P.dpc_se_a_tab_bwd(0, P.DPC_F64, 2, 1, [5], 8, None, f64(8), i32(2), i32(10), f64(40),
                           f64(64), f64(40))
    with pytest.raises(ValueError, match="GPU"):
        P.dpc_env_mat_a(0, P.DPC_F64, 2, 1, 5, 20.0, 6.0, 0.5, [0.0], [1.0], [1.0], f64(6), i32(2),
                        i32(10), f64(40))
    with pytest.raises(ValueError, match="GPU"):
        P.dpc_nlist_reverse(0, 2, 1, [5], 20.0, f64(6), i32(2), i32(10), i32(10))
    with pytest.raises(ValueError, match="GPU"):
        P.dpc_force_a(0, P.DPC_F64, 2, 1, 5, 20.0, 6.0, 0.5, [1.0], [1.0], f64(6), i32(2), i32(10),
                      i32(10), f64(40), f64(6), f64(18))
    net = P.dpc_fitting_net()
    net.n_in, net.width = 16, 8
    with pytest.raises(ValueError, match="GPU"):
        P.dpc_fitting_fwd_bwd(0, 1, 4, net, f64(64), f64(1000), 8000, f64(4))


def test_nlist_entry_point_validates_before_launch():
    fake = 4096
    nb = P.dpc_nlist_workspace_bytes(100, 20.0, 5.0)
    assert nb > 100 * 32 and nb % 256 == 0
    assert P.dpc_nlist_workspace_bytes(100, 10.0, 5.0) == 0       # box not above 2 rc
    assert P.dpc_nlist_workspace_bytes(-1, 20.0, 5.0) == 0
    base = dict(stream=0, nloc=100, ntypes=2, sel=[8, 8], box=20.0, rc=5.0, coord=fake, atype=fake,
                workspace=fake * 256, workspace_bytes=nb, nlist=fake, wait=False)
    cases = [(dict(box=10.0), B.DPC_ERANGE), (dict(rc=0.0), B.DPC_ERANGE), (dict(rc=float("nan")), B.DPC_ERANGE),
             (dict(nloc=-1), B.DPC_EINVAL), (dict(sel=[8, -1]), B.DPC_EINVAL), (dict(coord=0), B.DPC_EINVAL),
             (dict(workspace_bytes=nb - 1), B.DPC_EINVAL), (dict(workspace=fake * 256 + 16), B.DPC_EINVAL),
             (dict(ntypes=9, sel=[1] * 9), B.DPC_ENOTSUP), (dict(nlist=0), B.DPC_EINVAL),
             (dict(nloc=(1 << 28) + 1), B.DPC_ENOTSUP)]     # neighbour indices take 28 bits
    for kw, code in cases:
        a = dict(base); a.update(kw)
        with pytest.raises(P.DpcError) as e:
            P.dpc_nlist_build(**a)
        assert e.value.status == code, kw
    assert P.dpc_nlist_build(**{**base, "nloc": 0, "coord": 0, "nlist": 0, "wait": True}) == (0, 0)
