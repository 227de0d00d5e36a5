"""Environment matrix R~ and force / virial assembly (oracle).

Paper Sec. II: for neighbour j of atom i with r_ij = r_j - r_i (here the
minimum image in a cubic periodic box) and r = |r_ij|, the weighting function
of Eq. (1) is

    s(r) = 1/r                                   r < r_cs
         = (1/r) [u^3 (-6 u^2 + 15 u - 10) + 1]  r_cs <= r < r_c,  u = (r - r_cs) / (r_c - r_cs)
         = 0                                     r >= r_c,

and the row of R~ is (s, s x, s y, s z) normalised per centre type t: the
first element as (s - mean_t) / sigma_t, the other three divided by
sigma_all_t (the normalisation equations after Eq. (1)).  Padding rows are
zero.

Forces are F = -dE/dr.  Given dE/dR~ (the backward pass of the descriptor),
each valid pair contributes g_ij = dE/dr_ij = sum_c dE/dR~_ij[c] dR~_ij[c]/dr_ij;
since r_ij = r_j - r_i, F_i gets +g_ij and F_j gets -g_ij.  The per-atom
virial of atom i is V_i = -sum_j r_ij (x) g_ij (V[a][b] = -sum r_a g_b), so
that sum_i V_i[a][b] = -dE/d eps_ba for the homogeneous deformation
r_ij -> (1 + eps) r_ij.

Test infrastructure: plain float64 numpy, no blocking or fusion.
"""
import numpy as np


def weight(r, rc, rcs):
    """s(r) and ds/dr (Eq. (1)), elementwise."""
    r = np.asarray(r, float)
    s = np.zeros_like(r)
    ds = np.zeros_like(r)
    inner = r < rcs
    mid = (r >= rcs) & (r < rc)
    s[inner] = 1.0 / r[inner]
    ds[inner] = -1.0 / r[inner] ** 2
    rm = r[mid]
    u = (rm - rcs) / (rc - rcs)
    sw = u ** 3 * (-6.0 * u ** 2 + 15.0 * u - 10.0) + 1.0
    dsw = (-30.0 * u ** 4 + 60.0 * u ** 3 - 30.0 * u ** 2) / (rc - rcs)
    s[mid] = sw / rm
    ds[mid] = dsw / rm - sw / rm ** 2
    return s, ds


def pair_vectors(coords, box, nlist, atoms=None):
    """r_ij = r_j - r_i, minimum image in a cubic box of edge ``box``; zero
    for padding slots.  [n, nnei, 3]; row n of ``nlist`` belongs to atom
    ``atoms[n]`` (default: atom n)."""
    n, nnei = nlist.shape
    atoms = np.arange(n) if atoms is None else np.asarray(atoms)
    rij = np.zeros((n, nnei, 3))
    for row in range(n):
        i = atoms[row]
        for s in range(nnei):
            j = nlist[row, s]
            if j < 0:
                continue
            d = coords[j] - coords[i]
            d = d - box * np.round(d / box)
            rij[row, s] = d
    return rij


def rows_from_vectors(rij, valid, atype, rc, rcs, mean, sigma, sigma_all):
    """Normalised rows of R~ from pair vectors (valid [n, nnei] bool)."""
    r = np.sqrt(np.sum(rij * rij, axis=-1))
    s, _ = weight(np.where(valid, r, rc), rc, rcs)
    t = atype[:, None]
    em = np.zeros(rij.shape[:2] + (4,))
    em[..., 0] = (s - mean[t]) / sigma[t]
    em[..., 1:] = (s[..., None] * rij) / sigma_all[t][..., None]
    em[~valid] = 0.0
    return em


def env_mat(coords, box, atype, nlist, rc, rcs, mean, sigma, sigma_all, atoms=None):
    """R~ [n, nnei, 4] of atoms 0..n-1, or of ``atoms`` (then ``atype`` and
    ``nlist`` are those atoms' rows)."""
    rij = pair_vectors(coords, box, nlist, atoms)
    return rows_from_vectors(rij, nlist >= 0, atype, rc, rcs, mean, sigma, sigma_all)


def pair_gradients(rij, valid, atype, rc, rcs, sigma, sigma_all, dE_dem):
    """g_ij = sum_c dE/dR~_ij[c] dR~_ij[c]/dr_ij  [n, nnei, 3]:
    d(s)/dr_ij = s'(r) r_ij / r, d(s x_a)/dr_b = s'(r) x_a x_b / r + s delta_ab."""
    n, nnei = valid.shape
    g = np.zeros((n, nnei, 3))
    for i in range(n):
        t = atype[i]
        for sl in range(nnei):
            if not valid[i, sl]:
                continue
            x = rij[i, sl]
            r = np.sqrt(np.dot(x, x))
            s, ds = weight(np.array([r]), rc, rcs)
            s, ds = s[0], ds[0]
            lam = dE_dem[i, sl]
            grad = lam[0] / sigma[t] * ds * x / r
            for a in range(3):
                grad = grad + lam[1 + a] / sigma_all[t] * (ds * x[a] * x / r + s * np.eye(3)[a])
            g[i, sl] = grad
    return g


def force_virial(coords, box, atype, nlist, rc, rcs, mean, sigma, sigma_all, dE_dem):
    """Forces F [n, 3] and per-atom virials V [n, 3, 3] from dE/dR~."""
    valid = nlist >= 0
    rij = pair_vectors(coords, box, nlist)
    g = pair_gradients(rij, valid, atype, rc, rcs, sigma, sigma_all, dE_dem)
    n = nlist.shape[0]
    F = np.zeros((n, 3))
    V = np.zeros((n, 3, 3))
    for i in range(n):
        for sl in np.nonzero(valid[i])[0]:
            j = nlist[i, sl]
            F[i] += g[i, sl]
            F[j] -= g[i, sl]
            V[i] -= np.outer(rij[i, sl], g[i, sl])
    return F, V
