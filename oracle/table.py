"""Piecewise fifth-order Hermite tabulation of the embedding net (oracle).

Paper Sec. II, the paragraph on the compression of the embedding net: the input
range is cut into equal intervals of width Delta t; on [x_l, x_{l+1}) each
channel m is replaced by

    g_m^l(t) = a t^5 + b t^4 + c t^3 + d t^2 + e t + f,     t = x - x_l,

whose six coefficients are fixed by the value, first and second derivative
of G_m at both interval ends (the constraint equations), giving the closed
forms for a..f printed right after them, with h = y_{l+1} - y_l.

Reading of the paper (listed in the design notes):
* the polynomial variable is the offset t = x - x_l from the left node: only
  then are d = y''_l / 2, e = y'_l, f = y_l the right low-order coefficients;
* the tabulated range is [lo, x_up] with lo = s^(r_c) and x_up = lo + L1*d1
  the first node above the largest observed s^; an extrapolation band
  [x_up, x_end], x_end = x_up + L2*d2, uses the coarser stride d2;
* interval index l = floor((x - lo) / d1) (left-closed intervals), clamped
  into the range; inputs below lo use interval 0 with t < 0; inputs at or
  beyond x_end are clamped to the last node: g = value there, g' = g'' = 0.
"""
import numpy as np

from .net import embed_d2


def hermite_coefficients(y0, dy0, d2y0, y1, dy1, d2y1, dt):
    """(a, b, c, d, e, f) of the quintic matching (y, y', y'') at both ends of
    an interval of width dt -- the paper's closed forms, verbatim."""
    h = y1 - y0
    a = (12.0 * h - 6.0 * (dy1 + dy0) * dt + (d2y1 - d2y0) * dt ** 2) / (2.0 * dt ** 5)
    b = (-30.0 * h + (14.0 * dy1 + 16.0 * dy0) * dt + (3.0 * d2y0 - 2.0 * d2y1) * dt ** 2) / (2.0 * dt ** 4)
    c = (20.0 * h - (8.0 * dy1 + 12.0 * dy0) * dt - (3.0 * d2y0 - d2y1) * dt ** 2) / (2.0 * dt ** 3)
    d = 0.5 * d2y0
    e = dy0
    f = y0
    return a, b, c, d, e, f


class Table:
    """Hermite table of one embedding net.

    ``coef`` has shape [L1 + L2, M, 6] holding (f, e, d, c, b, a), i.e. the
    coefficients in ascending powers of t."""

    def __init__(self, lo, d1, L1, d2, L2, coef):
        self.lo, self.d1, self.L1 = float(lo), float(d1), int(L1)
        self.d2, self.L2 = float(d2), int(L2)
        self.coef = coef

    @property
    def M(self):
        return self.coef.shape[1]

    @property
    def x_up(self):
        return self.lo + self.L1 * self.d1

    @property
    def x_end(self):
        return self.x_up + self.L2 * self.d2

    def rounded(self, dtype):
        """Copy whose coefficients are rounded to ``dtype`` (kept as float64)."""
        return Table(self.lo, self.d1, self.L1, self.d2, self.L2,
                     self.coef.astype(dtype).astype(np.float64))

    def locate(self, x):
        """Interval index l, local offset t and the clamp flag for inputs x."""
        x = np.asarray(x, np.float64)
        x_up, x_end = self.x_up, self.x_end
        main = x < x_up
        band = (~main) & (x < x_end)
        l_main = np.clip(np.floor((x - self.lo) / self.d1), 0, self.L1 - 1)
        l_band = np.clip(np.floor((x - x_up) / self.d2), 0, self.L2 - 1)
        t_main = x - (self.lo + l_main * self.d1)
        t_band = x - (x_up + l_band * self.d2)
        l = np.where(main, l_main, np.where(band, self.L1 + l_band, self.L1 + self.L2 - 1))
        t = np.where(main, t_main, np.where(band, t_band, self.d2))
        clamped = ~(main | band)
        return l.astype(np.int64), t, clamped

    def evaluate(self, x, order=1):
        """g, g' (and g'' if order == 2) for inputs x [n]; each [n, M]."""
        l, t, clamped = self.locate(x)
        c = self.coef[l]                      # [n, M, 6]
        t = t[:, None]
        f, e, d, cc, b, a = (c[..., k] for k in range(6))
        g = ((((a * t + b) * t + cc) * t + d) * t + e) * t + f
        g1 = (((5.0 * a * t + 4.0 * b) * t + 3.0 * cc) * t + 2.0 * d) * t + e
        g1 = np.where(clamped[:, None], 0.0, g1)
        if order == 1:
            return g, g1
        g2 = ((20.0 * a * t + 12.0 * b) * t + 6.0 * cc) * t + 2.0 * d
        g2 = np.where(clamped[:, None], 0.0, g2)
        return g, g1, g2


def nodes(lo, d1, L1, d2, L2):
    """Main nodes lo + l*d1 (l = 0..L1) and band nodes x_up + l*d2 (l = 0..L2)."""
    x_up = lo + L1 * d1
    main = np.array([lo + l * d1 for l in range(L1 + 1)])
    band = np.array([x_up + l * d2 for l in range(L2 + 1)])
    return main, band


def build_table_from(func, lo, d1, L1, d2, L2):
    """Tabulate a vector function given as ``func(x) -> (y, y', y'')`` (each
    [n, M]) on [lo, x_up] (stride d1) and on the band (stride d2)."""
    main, band = nodes(lo, d1, L1, d2, L2)
    parts = []
    for xs, dt in ((main, d1), (band, d2)):
        y, dy, d2y = func(xs)
        a, b, c, d, e, f = hermite_coefficients(y[:-1], dy[:-1], d2y[:-1],
                                                y[1:], dy[1:], d2y[1:], dt)
        parts.append(np.stack([f, e, d, c, b, a], axis=-1))   # [L, M, 6]
    return Table(lo, d1, L1, d2, L2, np.concatenate(parts, 0))


def build_table(net, lo, d1, L1, d2, L2):
    """Tabulate the embedding net ``net``."""
    return build_table_from(lambda x: embed_d2(x, net), lo, d1, L1, d2, L2)


def build_tables(inputs):
    """One table per ordered type pair alpha*ntypes+beta of a ``synth.Inputs``."""
    return [build_table(inputs.nets[p], inputs.lo[p], inputs.d1, int(inputs.L1[p]),
                        inputs.d2, int(inputs.L2[p])) for p in range(inputs.npair)]
