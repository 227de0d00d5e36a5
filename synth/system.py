"""Seeded structure, neighbour list and environment-matrix generator.

Every atom sits at a lattice *site* plus a bounded displacement (Gaussian
jitter for the metals, the rigid-molecule geometry for water).  Neighbour
candidates of an atom are therefore a fixed list of site offsets (the sites
within r_c + 2 * max|displacement|), which makes the search exact and cheap
even for 10^6 atoms.  Periodic images are folded by index arithmetic, and the
pair vector is the site offset plus the displacement difference.

R~ follows the paper's construction (Sec. II): the weighting function s(r)
of Eq. (1), the 4-vector (s, s*x, s*y, s*z) with (x, y, z) = r_j - r_i, then
s is shifted by its mean and divided by its standard deviation while the
three spatial components are divided by one pooled standard deviation
sigma_all.  The statistics are taken per centre type over the valid rows of
the generated structure itself (the paper takes them from training data,
which is not available).  Rows are blocked by neighbour type (sel_alpha slots
each), sorted by distance inside a block and zero-padded; padding slots hold
nlist = -1.
"""
from dataclasses import dataclass, field
from typing import List, Dict

import numpy as np

from .configs import Config

_SEED_ROOT = 210702103
_R_OH = 0.9572                 # Angstrom
_THETA_HOH = np.deg2rad(104.52)


@dataclass
class Inputs:
    cfg: Config
    atype: np.ndarray            # int32 [nloc]
    nlist: np.ndarray            # int32 [nloc, nnei], -1 = padding
    em: np.ndarray               # float64 [nloc, nnei, 4]  (R~)
    nets: List[Dict]             # per ordered pair alpha*ntypes+beta: {"W": [..], "b": [..]}
    lo: np.ndarray               # float64 [npair]  lower end of the table (s^ at r_c)
    L1: np.ndarray               # int64 [npair]    intervals of stride d1
    L2: np.ndarray               # int64 [npair]    intervals of stride d2 (extrapolation band)
    s_hat_max: np.ndarray        # float64 [npair]  largest observed s^ (nan if no pairs)
    stats: Dict                  # per centre type: mean, sigma, sigma_all
    dT: np.ndarray = None        # float64 [nloc, m1, 4] upstream gradient dE/dT
    n_valid: int = 0
    coords: np.ndarray = None    # float64 [nloc, 3] positions (cubic periodic box of edge cfg.box)

    @property
    def d1(self) -> float:
        return self.cfg.d1

    @property
    def d2(self) -> float:
        return self.cfg.d2

    @property
    def npair(self) -> int:
        return self.cfg.ntypes ** 2


def _rngs(cfg: Config):
    ss = np.random.SeedSequence([_SEED_ROOT, cfg.seed])
    pos, species, orient, nets, grad = ss.spawn(5)
    return (np.random.default_rng(pos), np.random.default_rng(species),
            np.random.default_rng(orient), np.random.default_rng(nets),
            np.random.default_rng(grad))


def _random_rotations(rng, n):
    """Uniform random rotation matrices from unit quaternions, [n, 3, 3]."""
    q = rng.standard_normal((n, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    w, x, y, z = q.T
    R = np.empty((n, 3, 3))
    R[:, 0, 0] = 1 - 2 * (y * y + z * z)
    R[:, 0, 1] = 2 * (x * y - z * w)
    R[:, 0, 2] = 2 * (x * z + y * w)
    R[:, 1, 0] = 2 * (x * y + z * w)
    R[:, 1, 1] = 1 - 2 * (x * x + z * z)
    R[:, 1, 2] = 2 * (y * z - x * w)
    R[:, 2, 0] = 2 * (x * z - y * w)
    R[:, 2, 1] = 2 * (y * z + x * w)
    R[:, 2, 2] = 1 - 2 * (x * x + y * y)
    return R


def _structure(cfg: Config, rng_pos, rng_species, rng_orient):
    """Return (basis sites [nb,3], types [natoms], disp [natoms,3])."""
    N = cfg.ncell
    ncells = N ** 3
    L = cfg.cell_edge
    if cfg.kind == "fcc":
        basis = L * np.array([[0, 0, 0], [0.5, 0.5, 0], [0.5, 0, 0.5], [0, 0.5, 0.5]], float)
        nat = 4 * ncells
        disp = rng_pos.normal(0.0, cfg.jitter, size=(nat, 3)) if cfg.jitter > 0 else np.zeros((nat, 3))
        p = np.asarray(cfg.type_probs, float)
        if len(p) == 1:
            types = np.zeros(nat, np.int32)
        else:
            types = rng_species.choice(len(p), size=nat, p=p / p.sum()).astype(np.int32)
        return basis, types, disp
    if cfg.kind == "water":
        basis = np.zeros((3, 3))  # O, H1, H2 share the molecular site
        h = 0.5 * _THETA_HOH
        ref = np.array([[0.0, 0.0, 0.0],
                        [_R_OH * np.sin(h), 0.0, _R_OH * np.cos(h)],
                        [-_R_OH * np.sin(h), 0.0, _R_OH * np.cos(h)]])
        rot = _random_rotations(rng_orient, ncells)
        disp = np.einsum("nij,aj->nai", rot, ref).reshape(3 * ncells, 3)
        types = np.tile(np.array([0, 1, 1], np.int32), ncells)
        return basis, types, disp
    raise ValueError(cfg.kind)


def _candidate_offsets(basis, L, cut):
    """For each basis b: int array [ncand, 4] of (dx, dy, dz, b') with site
    distance < cut, excluding the atom itself."""
    nb = len(basis)
    K = int(np.ceil(cut / L)) + 1
    rng = np.arange(-K, K + 1)
    dc = np.stack(np.meshgrid(rng, rng, rng, indexing="ij"), -1).reshape(-1, 3)
    out = []
    for b in range(nb):
        rows = []
        for bp in range(nb):
            vec = dc * L + basis[bp] - basis[b]
            d = np.linalg.norm(vec, axis=1)
            keep = d < cut
            if bp == b:
                keep &= np.any(dc != 0, axis=1)
            sel = dc[keep]
            rows.append(np.concatenate([sel, np.full((len(sel), 1), bp)], 1))
        out.append(np.concatenate(rows, 0).astype(np.int64))
    return out


def weighting(r, rc, rcs):
    """s(r) of the paper's Eq. (1): 1/r inside r_cs, a C^2 quintic switch
    between r_cs and r_c, zero beyond."""
    r = np.asarray(r, float)
    u = (r - rcs) / (rc - rcs)
    sw = u * u * u * (-6.0 * u * u + 15.0 * u - 10.0) + 1.0
    with np.errstate(divide="ignore"):
        inv = 1.0 / r
    return np.where(r < rcs, inv, np.where(r < rc, inv * sw, 0.0))


def random_net(rng, widths):
    """Embedding-net weights W_k ~ N(0, 1/fan_in), b_k ~ N(0, 1)."""
    W, b = [], []
    for k in range(len(widths) - 1):
        fi, fo = widths[k], widths[k + 1]
        W.append(rng.normal(0.0, 1.0 / np.sqrt(fi), size=(fi, fo)))
        b.append(rng.normal(0.0, 1.0, size=(fo,)))
    return {"W": W, "b": b}


def _chunk(cfg, basis, types, disp, sel, sel_off, cand, b, c0, c1, nlist, em):
    """Neighbour search + raw 4-vectors for the atoms of basis ``b`` in cells
    [c0, c1); writes their nlist/em rows and returns partial statistics."""
    N, L, nb, nt, nnei = cfg.ncell, cfg.cell_edge, len(basis), cfg.ntypes, int(sel.sum())
    dxyz, bp = cand[:, :3], cand[:, 3]
    site_vec = dxyz * L + basis[bp] - basis[b]
    cells = np.arange(c0, c1)
    cx, cy, cz = cells // (N * N), (cells // N) % N, cells % N
    j = ((((cx[:, None] + dxyz[None, :, 0]) % N) * N
          + (cy[:, None] + dxyz[None, :, 1]) % N) * N
         + (cz[:, None] + dxyz[None, :, 2]) % N) * nb + bp[None, :]
    rows = slice(c0 * nb + b, c1 * nb, nb)      # atoms of basis b in these cells
    vec = site_vec[None, :, :] + disp[j] - disp[rows][:, None, :]
    r = np.sqrt(np.einsum("ncd,ncd->nc", vec, vec))
    valid = r < cfg.rc
    tj = types[j]
    ti = types[rows]
    nc = len(cells)
    cnt = np.stack([(valid & (tj == beta)).sum(1) for beta in range(nt)], 1)  # [nc, nt]
    if (cnt > sel[None, :]).any():
        raise ValueError(f"{cfg.name}: neighbour count {cnt.max(0)} exceeds sel={tuple(sel)}")
    stats = np.zeros((nt, 5))                    # s_sum, s_sq, n, v_sum, v_sq per centre type
    smax = np.full((nt, nt), -np.inf)
    kmax = int(cnt.sum(1).max()) if nc else 0
    if kmax == 0:
        return stats, smax, 0
    # one sort: type-major, distance-minor, invalid candidates last
    key = np.where(valid, tj * (4.0 * cfg.rc) + r, np.inf)
    order = np.argsort(key, axis=1, kind="stable")[:, :kmax]
    rs = np.take_along_axis(r, order, 1)
    js = np.take_along_axis(j, order, 1)
    ts = np.take_along_axis(tj, order, 1)
    vs = np.take_along_axis(vec, order[:, :, None], 1)
    q = np.arange(kmax)[None, :]
    ok = q < cnt.sum(1)[:, None]
    start = np.concatenate([np.zeros((nc, 1), np.int64), np.cumsum(cnt, 1)[:, :-1]], 1)
    col = np.where(ok, sel_off[ts] + q - np.take_along_axis(start, ts, 1), nnei)
    s = np.where(ok, weighting(np.where(ok, rs, cfg.rc), cfg.rc, cfg.rcs), 0.0)
    vals = np.concatenate([s[:, :, None], s[:, :, None] * vs], 2)
    nl_blk = np.full((nc, nnei + 1), -1, np.int32)
    em_blk = np.zeros((nc, nnei + 1, 4))
    np.put_along_axis(nl_blk, col, np.where(ok, js, -1).astype(np.int32), 1)
    np.put_along_axis(em_blk, col[:, :, None], vals, 1)
    nlist[rows] = nl_blk[:, :nnei]
    em[rows] = em_blk[:, :nnei]
    # statistics per centre type; s is largest at the first slot of each block
    v = vals[:, :, 1:]
    per_row = np.stack([s.sum(1), (s * s).sum(1), ok.sum(1),
                        v.sum((1, 2)), (v * v).sum((1, 2))], 1)
    for alpha in range(nt):
        ra = ti == alpha
        if not ra.any():
            continue
        stats[alpha] = per_row[ra].sum(0)
        for beta in range(nt):
            has = ra & (cnt[:, beta] > 0)
            if has.any():
                first = np.take_along_axis(em_blk[:, :, 0], np.full((nc, 1), sel_off[beta]), 1)[:, 0]
                smax[alpha, beta] = first[has].max()
    return stats, smax, int(ok.sum())


def random_fitting_net(rng, n_in, widths=(240, 240, 240)):
    """Fitting-net weights (descriptor -> energy): hidden layers W_l ~
    N(0, 1/fan_in), b_l ~ N(0, 1); output w_out ~ N(0, 1/width), b_out ~ N(0, 1)."""
    W, b = [], []
    fan = n_in
    for w in widths:
        W.append(rng.normal(0.0, 1.0 / np.sqrt(fan), size=(fan, w)))
        b.append(rng.normal(0.0, 1.0, size=(w,)))
        fan = w
    return {"W": W, "b": b, "w_out": rng.normal(0.0, 1.0 / np.sqrt(fan), size=(fan,)),
            "b_out": float(rng.normal(0.0, 1.0))}


def random_grad(rng, nat, m1, threads=None, chunk=65536, width=4):
    """dE/dT ~ N(0, 1) of shape [nat, m1, width] (width 4: dE/dT; width M':
    dE/dD, or a T-shaped input of the descriptor backward), drawn in fixed
    chunks of atoms from streams spawned off ``rng`` (deterministic for any
    thread count)."""
    from concurrent.futures import ThreadPoolExecutor
    import os
    out = np.empty((nat, m1, width))
    starts = list(range(0, nat, chunk))
    seeds = rng.bit_generator.seed_seq.spawn(len(starts))
    threads = threads or max(1, min(16, len(os.sched_getaffinity(0))))

    def run(k):
        a0 = starts[k]
        a1 = min(nat, a0 + chunk)
        out[a0:a1] = np.random.default_rng(seeds[k]).standard_normal((a1 - a0, m1, width))

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(run, range(len(starts))))
    return out


def make_inputs(cfg: Config, chunk_cells: int = 2048, with_grad: bool = True,
                threads: int = None, verbose: bool = False) -> Inputs:
    """Build the full seeded input set for ``cfg`` (float64 R~).

    The work is split into fixed chunks of cells; chunks run on a thread pool
    but their partial statistics are reduced in chunk order, so the result is
    independent of the thread count."""
    from concurrent.futures import ThreadPoolExecutor
    import os
    rng_pos, rng_species, rng_orient, rng_nets, rng_grad = _rngs(cfg)
    basis, types, disp = _structure(cfg, rng_pos, rng_species, rng_orient)
    N, L = cfg.ncell, cfg.cell_edge
    nb = len(basis)
    nat = len(types)
    nt = cfg.ntypes
    sel = np.asarray(cfg.sel, np.int64)
    sel_off = np.concatenate([[0], np.cumsum(sel)])
    nnei = int(sel.sum())
    dmax = float(np.max(np.linalg.norm(disp, axis=1))) if nat else 0.0
    cut = cfg.rc + 2.0 * dmax + 1e-9
    if cfg.box < 2.0 * cut:
        raise ValueError(f"{cfg.name}: box {cfg.box:.3f} too small for candidate cutoff {cut:.3f}")
    cands = _candidate_offsets(basis, L, cut)

    nlist = np.empty((nat, nnei), np.int32)
    em = np.empty((nat, nnei, 4), np.float64)
    ncells = N ** 3
    tasks = [(b, c0, min(ncells, c0 + chunk_cells)) for b in range(nb)
             for c0 in range(0, ncells, chunk_cells)]
    if threads is None:
        threads = max(1, min(16, len(os.sched_getaffinity(0))))

    def run(t):
        b, c0, c1 = t
        out = _chunk(cfg, basis, types, disp, sel, sel_off, cands[b], b, c0, c1, nlist, em)
        if verbose:
            print(f"  {cfg.name}: basis {b} cells {c0}..{c1 - 1}", flush=True)
        return out

    with ThreadPoolExecutor(threads) as ex:
        parts = list(ex.map(run, tasks))
    stats = np.zeros((nt, 5))
    s_max = np.full((nt, nt), -np.inf)
    n_valid = 0
    for st, sm, nv in parts:                     # fixed order -> deterministic sums
        stats += st
        s_max = np.maximum(s_max, sm)
        n_valid += nv

    # normalisation (per centre type), padding rows stay exactly zero
    mean = np.zeros(nt); sig = np.ones(nt); sig_all = np.ones(nt)
    for alpha in range(nt):
        s_sum, s_sq, n, v_sum, v_sq = stats[alpha]
        if n > 0:
            mean[alpha] = s_sum / n
            var = s_sq / n - mean[alpha] ** 2
            sig[alpha] = np.sqrt(var) if var > 0 else 1.0
            vm = v_sum / (3 * n)
            vvar = v_sq / (3 * n) - vm * vm
            sig_all[alpha] = np.sqrt(vvar) if vvar > 0 else 1.0

    def norm(a0):
        sl = slice(a0, min(nat, a0 + 16384))
        valid = nlist[sl] >= 0
        ta = types[sl]
        e = em[sl]
        e[:, :, 0] = np.where(valid, (e[:, :, 0] - mean[ta][:, None]) / sig[ta][:, None], 0.0)
        e[:, :, 1:] /= sig_all[ta][:, None, None]

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(norm, range(0, nat, 16384)))

    # tabulation range per ordered pair: [s^(r_c), max observed s^] (paper Sec. II)
    npair = nt * nt
    lo = np.zeros(npair); L1 = np.zeros(npair, np.int64); L2 = np.zeros(npair, np.int64)
    shmax = np.full(npair, np.nan)
    for alpha in range(nt):
        lo_a = (0.0 - mean[alpha]) / sig[alpha]
        for beta in range(nt):
            p = alpha * nt + beta
            lo[p] = lo_a
            if np.isfinite(s_max[alpha, beta]):
                shmax[p] = (s_max[alpha, beta] - mean[alpha]) / sig[alpha]
                L1[p] = int(np.floor((shmax[p] - lo_a) / cfg.d1)) + 1
            else:
                L1[p] = 1
            # extrapolation band as wide as the main range, stride d2
            L2[p] = max(1, int(np.ceil(L1[p] * cfg.d1 / cfg.d2)))

    nets = [random_net(rng_nets, cfg.widths) for _ in range(npair)]
    dT = random_grad(rng_grad, nat, cfg.m1, threads) if with_grad else None
    st = {"mean": mean, "sigma": sig, "sigma_all": sig_all, "dmax": dmax}
    # positions: cell c = i // nb at (c // N^2, (c // N) % N, c % N) * L, plus the basis site and displacement
    c = np.arange(nat) // nb
    cell = np.stack([c // (N * N), (c // N) % N, c % N], 1).astype(np.float64)
    coords = cell * L + basis[np.arange(nat) % nb] + disp
    return Inputs(cfg=cfg, atype=types.astype(np.int32), nlist=nlist, em=em, nets=nets,
                  lo=lo, L1=L1, L2=L2, s_hat_max=shmax, stats=st, dT=dT,
                  n_valid=n_valid, coords=coords)
