"""Forward and backward of the compressed se_a descriptor (oracle).

Paper Sec. II: rows of R~^i are blocked by neighbour type (sel_alpha slots
each, padding rows are zero); the embedding matrix G^i has rows
G_m(s^_ij), with s^_ij the first column of R~^i; S^i = (G^i)^T R~^i is M x 4,
S^i< holds its first M' rows, and D^i = S^i (S^i<)^T is M x M'.  In the
compressed model G_m is replaced by the tabulated quintic g_m and the product
is taken only over valid neighbours (the fused, padding-skipping kernel of
Sec. II).  T denotes S.

Backward (forces need derivatives of E w.r.t. R~, Sec. II): with
dT = dE/dT_i,

    dE/dR~_ij[k] = sum_m dT[m][k] g_m(x_ij)
                   + delta_{k0} sum_m g'_m(x_ij) sum_k' dT[m][k'] R~_ij[k'],

since x_ij = R~_ij[0] enters both through the row itself and through g.
Padding rows are not variables; their gradient is defined as 0.

Everything is evaluated atom by atom with the table evaluated on the valid
rows of one sel block at a time and a matmul for the contraction.
"""
import numpy as np

from .net import embed, embed_d2


def _blocks(sel):
    off = np.concatenate([[0], np.cumsum(sel)]).astype(np.int64)
    return [(beta, int(off[beta]), int(off[beta + 1])) for beta in range(len(sel))]


def forward(em, nlist, atype, tables, sel, m2, atoms=None, with_abs=False):
    """T [n, M, 4] and D [n, M, m2] for the atoms ``atoms`` (default: all).

    With ``with_abs`` also returns the abs-sum bounds used by the tolerances:
    A_T[m][k] = sum_j |g_m R~_jk| bounds the rounding of T (any summation
    order), and A_D[m][n] = sum_k A_T[m][k] |T[n][k]| + |T[m][k]| A_T[n][k]
    + |T[m][k] T[n][k]| bounds how an error of relative size eps in the terms
    of T (eps * A_T) and in the products of D propagates into D."""
    nt = len(sel)
    atoms = np.arange(nlist.shape[0]) if atoms is None else np.asarray(atoms)
    M = tables[0].M
    T = np.zeros((len(atoms), M, 4))
    AT = np.zeros_like(T) if with_abs else None
    for n, i in enumerate(atoms):
        for beta, s0, s1 in _blocks(sel):
            js = s0 + np.nonzero(nlist[i, s0:s1] >= 0)[0]
            if len(js) == 0:
                continue
            R = em[i, js]                                   # [nj, 4]
            g, _ = tables[atype[i] * nt + beta].evaluate(R[:, 0])   # [nj, M]
            T[n] += g.T @ R
            if with_abs:
                AT[n] += np.abs(g).T @ np.abs(R)
    D = T @ np.transpose(T[:, :m2, :], (0, 2, 1))
    if not with_abs:
        return T, D
    aT = np.abs(T)
    AD = (AT @ np.transpose(aT[:, :m2, :], (0, 2, 1)) + aT @ np.transpose(AT[:, :m2, :], (0, 2, 1))
          + aT @ np.transpose(aT[:, :m2, :], (0, 2, 1)))
    return T, D, AT, AD


def backward(em, nlist, atype, tables, sel, dT, atoms=None, with_abs=False):
    """dE/dR~ [n, nnei, 4] for the atoms ``atoms`` (default: all), given
    dT = dE/dT [nloc, M, 4] (indexed by the same atoms)."""
    nt = len(sel)
    atoms = np.arange(nlist.shape[0]) if atoms is None else np.asarray(atoms)
    dR = np.zeros((len(atoms),) + em.shape[1:])
    AR = np.zeros_like(dR) if with_abs else None
    for n, i in enumerate(atoms):
        dTi = dT[i]                                         # [M, 4]
        for beta, s0, s1 in _blocks(sel):
            js = s0 + np.nonzero(nlist[i, s0:s1] >= 0)[0]
            if len(js) == 0:
                continue
            R = em[i, js]
            g, gp = tables[atype[i] * nt + beta].evaluate(R[:, 0])
            w = R @ dTi.T                                   # [nj, M]: sum_k dT[m][k] R[k]
            dR[n, js] = g @ dTi
            dR[n, js, 0] += np.sum(gp * w, axis=1)
            if with_abs:
                AR[n, js] = np.abs(g) @ np.abs(dTi)
                AR[n, js, 0] += np.sum(np.abs(gp) * (np.abs(R) @ np.abs(dTi).T), axis=1)
    return (dR, AR) if with_abs else dR


def forward_untabulated(em, nlist, atype, nets, sel, m2, atoms=None):
    """The original (uncompressed) path: G from the real embedding net,
    materialised as a matrix and multiplied by R~ -- used to pin the
    tabulated forward on small inputs."""
    nt = len(sel)
    atoms = np.arange(nlist.shape[0]) if atoms is None else np.asarray(atoms)
    M = nets[0]["W"][-1].shape[1]
    T = np.zeros((len(atoms), M, 4))
    for n, i in enumerate(atoms):
        for beta, s0, s1 in _blocks(sel):
            js = s0 + np.nonzero(nlist[i, s0:s1] >= 0)[0]
            if len(js) == 0:
                continue
            R = em[i, js]
            G = embed(R[:, 0], nets[atype[i] * nt + beta])
            T[n] += G.T @ R
    D = T @ np.transpose(T[:, :m2, :], (0, 2, 1))
    return T, D


def backward_untabulated(em, nlist, atype, nets, sel, dT, atoms=None):
    """dE/dR~ through the original (uncompressed) embedding net: the backward
    formula of this module with g, g' replaced by G and G' of the net (its
    forward-mode first derivative) -- the reference of the table-stride
    study on small inputs."""
    nt = len(sel)
    atoms = np.arange(nlist.shape[0]) if atoms is None else np.asarray(atoms)
    dR = np.zeros((len(atoms),) + em.shape[1:])
    for n, i in enumerate(atoms):
        dTi = dT[i]
        for beta, s0, s1 in _blocks(sel):
            js = s0 + np.nonzero(nlist[i, s0:s1] >= 0)[0]
            if len(js) == 0:
                continue
            R = em[i, js]
            G, Gp, _ = embed_d2(R[:, 0], nets[atype[i] * nt + beta])
            dR[n, js] = G @ dTi
            dR[n, js, 0] += np.sum(Gp * (R @ dTi.T), axis=1)
    return dR


def descriptor_backward(T, dD):
    """dE/dT [n, M, 4] from dE/dD [n, M, M'] (Sec. II: D_i = T_i (T_i<)^T,
    T_i< the first M' rows of T_i).  D[m][n] = sum_k T[m][k] T[n][k] holds
    T twice, once through row m and once through row n < M', so

        dE/dT[m][k] = sum_{n<M'} dE/dD[m][n] T[n][k]
                      + (m < M') sum_{m'} dE/dD[m'][m] T[m'][k].

    Written as two explicit loops over the atom's entries."""
    n_at, M, m2 = dD.shape
    dT = np.zeros((n_at, M, 4))
    for a in range(n_at):
        for m in range(M):
            for k in range(4):
                v = 0.0
                for n in range(m2):
                    v += dD[a, m, n] * T[a, n, k]
                if m < m2:
                    for q in range(M):
                        v += dD[a, q, m] * T[a, q, k]
                dT[a, m, k] = v
    return dT


def energy(T, lam):
    """Scalar E = sum <Lambda_i, T_i> whose dE/dT is Lambda (FD pins)."""
    return float(np.sum(T * lam))
