"""Helpers of the GPU parity tests: the oracle's view of a workload's inputs
and the comparisons (per-atom normwise and abs-sum-scaled componentwise).
The oracle side always starts from the same seeded inputs (``synth``) and
builds its own tables."""
import numpy as np

from oracle import cref
from oracle.se_a import backward as np_backward
from oracle.se_a import forward as np_forward
from oracle.table import build_tables as oracle_tables

TOL = {"f64": 1e-12, "f32": 1e-5, "f32acc64": 1e-5}


def oracle_view(inputs, atoms, dtype="f64"):
    """Oracle inputs for the rows ``atoms``: float64 arrays, rounded through
    float32 first for the float32 storage modes."""
    tabs = oracle_tables(inputs)
    em = inputs.em[atoms]
    dT = inputs.dT[atoms]
    if dtype != "f64":
        tabs = [t.rounded(np.float32) for t in tabs]
        em = em.astype(np.float32).astype(np.float64)
        dT = dT.astype(np.float32).astype(np.float64)
    return tabs, em, inputs.nlist[atoms], inputs.atype[atoms], dT


def normwise(got, ref):
    """max over atoms of ||got_i - ref_i||_inf / ||ref_i||_inf (atoms whose
    reference is all zero must match exactly)."""
    n = got.shape[0]
    d = np.abs(got - ref).reshape(n, -1).max(1)
    s = np.abs(ref).reshape(n, -1).max(1)
    if np.any((s == 0) & (d != 0)):
        return np.inf
    return float(np.max(np.where(s > 0, d / np.where(s > 0, s, 1), 0.0))) if n else 0.0


def oracle_fwd_bwd(inputs, atoms, dtype="f64"):
    tabs, em, nl, at, dT = oracle_view(inputs, atoms, dtype)
    pb = cref.Problem(em, nl, at, tabs, inputs.cfg.sel, inputs.cfg.m2)
    T, D = pb.forward()
    dR = pb.backward(dT)
    return T, D, dR


def oracle_abs_bounds(inputs, atoms, dtype="f64"):
    """Abs-sum bounds A_T, A_D, A_dR (numpy oracle) for componentwise checks."""
    tabs, em, nl, at, dT = oracle_view(inputs, atoms, dtype)
    _, _, AT, AD = np_forward(em, nl, at, tabs, inputs.cfg.sel, inputs.cfg.m2, with_abs=True)
    _, AR = np_backward(em, nl, at, tabs, inputs.cfg.sel, dT, with_abs=True)
    return AT, AD, AR


def compare(got, ref, bounds=None, tol=1e-12):
    """Parity report of (T, D, dR) against the oracle."""
    rep = {}
    for name, g, r in zip(("T", "D", "dR"), got, ref):
        rep[name + "_normwise"] = normwise(g, r)
    if bounds is not None:
        for name, g, r, a in zip(("T", "D", "dR"), got, ref, bounds):
            excess = np.abs(g - r) - tol * a
            rep[name + "_componentwise_ok"] = bool(np.all(excess <= 0))
    rep["ok"] = all(v <= tol for k, v in rep.items() if k.endswith("normwise")) and all(
        v for k, v in rep.items() if k.endswith("_ok"))
    return rep
