"""The no-allocation neighbour list (dpc_nlist_build_noalloc) against the
one with a caller's workspace (dpc_nlist_build): identical lists and status
counters on two calls in a row, the second on a smaller system, so that the
second call runs on the static cell list the first one left behind."""
import numpy as np
import pytest

from synth import make_inputs
from synth.configs import get_config

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _both(x, sel=None):
    import paper_2107_02103_amd as P
    c = x.cfg
    sel = c.sel if sel is None else sel
    n, nnei = len(x.coords), int(sum(sel))
    co = torch.from_numpy(x.coords).cuda()
    at = torch.from_numpy(x.atype).cuda()
    s = torch.cuda.current_stream()
    nb = P.dpc_nlist_workspace_bytes(n, c.box, c.rc)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    ref = torch.full((n, nnei), -7, dtype=torch.int32, device="cuda")
    P.dpc_nlist_build(s, n, c.ntypes, sel, c.box, c.rc, co, at, ws, nb, ref, wait=False)
    got = torch.full((n, nnei), -9, dtype=torch.int32, device="cuda")
    st = torch.full((2,), -1, dtype=torch.int32, device="cuda")
    P.dpc_nlist_build_noalloc(s, n, c.ntypes, sel, c.box, c.rc, co, at, got, st)
    torch.cuda.synchronize()
    return got.cpu().numpy(), st.cpu().numpy(), ref.cpu().numpy(), ws[:8].view(torch.int32).cpu().numpy()


def test_noalloc_matches_workspace_entry_point():
    for key, sel in (("alcumg32000", None), ("tiny_alloy", (10, 3, 3)), ("tiny_water", None)):
        x = make_inputs(get_config(key), with_grad=False)
        got, st, ref, st_ref = _both(x, sel)
        print(f"[no-alloc] {key} sel {sel or x.cfg.sel}: status {st.tolist()} vs {st_ref.tolist()}",
              flush=True)
        np.testing.assert_array_equal(got, ref)
        np.testing.assert_array_equal(st, st_ref)
    assert st_ref[0] == 0


def test_noalloc_refuses_too_many_atoms():
    import paper_2107_02103_amd as P
    n = P.DPC_NLIST_NOALLOC_MAX_ATOMS + 1
    with pytest.raises(P.DpcError) as e:
        P.dpc_nlist_build_noalloc(0, n, 1, [8], 1000.0, 5.0, 4096, 4096, 4096, None)
    assert e.value.status == P.DPC_ENOTSUP
