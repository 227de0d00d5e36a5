"""Hand-placed neighbour rows for edge cases of the tabulated descriptor.

Unlike ``synth.system`` these inputs come from no structure: every atom gets
a random subset of its slots, and the first column of each valid row
(s^ after normalisation) is placed in the four parts of the tabulation range
in fixed shares (paper Sec. II: the table covers [s^(r_c), s^(r_l)] with an
equal step; the extrapolation band and the clamp beyond it are a reading
where the paper is silent): below the lower end, in the main range, in the band, and past the
band's end, plus rows exactly on the range's boundaries and on nodes.  The
spatial columns are standard normal.  Only inputs are produced here.
"""
import numpy as np

from .configs import Config
from .system import Inputs, random_net

# share of valid rows in each part: [lo - 0.2 d1, lo), [lo, x_up), [x_up, x_end),
# [x_end, x_end + 0.5]; the rest sit exactly on lo, x_up, x_end or a node
SHARES = (0.05, 0.55, 0.25, 0.10)


def place_x(rng, n, lo, d1, L1, d2, L2):
    """n first-column values spread over the four parts in the SHARES
    proportions (rounded per part, the remainder on boundaries and nodes),
    in random order."""
    x_up = lo + L1 * d1
    x_end = x_up + L2 * d2
    counts = [int(np.floor(s * n)) for s in SHARES]
    parts = [rng.uniform(lo - 0.2 * d1, lo, counts[0]),
             rng.uniform(lo, x_up, counts[1]),
             rng.uniform(x_up, x_end, counts[2]),
             rng.uniform(x_end, x_end + 0.5, counts[3])]
    rest = n - sum(counts)
    # the ends of the parts, and the last doubles below x_up and x_end (whose
    # offsets from the part's origin can round up to a whole part)
    exact = np.concatenate([[lo, x_up, x_end, np.nextafter(x_up, -np.inf),
                             np.nextafter(x_end, -np.inf), np.nextafter(lo, np.inf)],
                            lo + rng.integers(1, L1, 8) * d1,
                            x_up + rng.integers(1, L2, 4) * d2])
    parts.append(exact[rng.integers(0, len(exact), rest)])
    x = np.concatenate(parts)
    return x[rng.permutation(n)]


def edge_inputs(nloc, sel, m1, m2, seed, lo=-0.6, L1=300, L2=30, d1=0.01, d2=0.1,
                fill=None):
    """Inputs (``synth.Inputs``) with random slot occupancy and first columns
    placed by ``place_x``; ``fill`` (0..1) fixes the share of valid slots per
    atom, else it is uniform in [0, 1]."""
    rng = np.random.default_rng(seed)
    nt = len(sel)
    cfg = Config("edge", "fcc", 1, rc=1.0, rcs=0.5, sel=tuple(sel), widths=(1, 8, 16, m1),
                 m2=m2, d1=d1, d2=d2)
    nnei = int(sum(sel))
    nlist = np.full((nloc, nnei), -1, np.int32)
    em = np.zeros((nloc, nnei, 4))
    for i in range(nloc):
        k = int(round(fill * nnei)) if fill is not None else int(rng.integers(0, nnei + 1))
        slots = rng.choice(nnei, size=k, replace=False)
        nlist[i, slots] = rng.integers(0, nloc, size=k)
        em[i, slots, 0] = place_x(rng, k, lo, d1, L1, d2, L2)
        em[i, slots, 1:] = rng.normal(size=(k, 3))
    atype = rng.integers(0, nt, size=nloc).astype(np.int32)
    nets = [random_net(rng, cfg.widths) for _ in range(nt * nt)]
    npair = nt * nt
    return Inputs(cfg=cfg, atype=atype, nlist=nlist, em=em, nets=nets, lo=np.full(npair, lo),
                  L1=np.full(npair, L1), L2=np.full(npair, L2), s_hat_max=np.zeros(npair),
                  stats={}, dT=rng.normal(size=(nloc, m1, 4)), n_valid=int((nlist >= 0).sum()))
