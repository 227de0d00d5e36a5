"""Embedding net G: s^ -> R^M and its derivatives (paper Sec. II).

The net maps the scalar s^ (first column of R~) to M channels through tanh
layers.  A layer whose output is twice as wide as its input adds the input
concatenated with itself ("residual doubling"); a layer of equal width adds
its input; otherwise there is no residual.

Derivatives are propagated in forward mode with x' = 1, x'' = 0:
    z = y W + b,            z' = y' W,          z'' = y'' W
    h = tanh(z),            h' = (1 - h^2) z',  h'' = (1 - h^2) z'' - 2 h (1 - h^2) z'^2
The paper only states that G' and G'' are cheap to evaluate (Sec. II, after
the coefficient formulas); this is the direct way.  Works for real and complex
arguments (complex input is used by the complex-step pins).
"""
import numpy as np


def _residual(y, fan_in, fan_out):
    if fan_out == 2 * fan_in:
        return np.concatenate([y, y], axis=-1)
    if fan_out == fan_in:
        return y
    return None


def embed(x, net):
    """G(x) for an array of inputs x [n] -> [n, M]."""
    y = np.asarray(x)[..., None]
    for W, b in zip(net["W"], net["b"]):
        h = np.tanh(y @ W + b)
        res = _residual(y, W.shape[0], W.shape[1])
        y = h if res is None else h + res
    return y


def embed_d2(x, net):
    """(G, G', G'') at x [n], each [n, M]."""
    y = np.asarray(x)[..., None]
    dy = np.ones_like(y)
    d2y = np.zeros_like(y)
    for W, b in zip(net["W"], net["b"]):
        z = y @ W + b
        dz = dy @ W
        d2z = d2y @ W
        h = np.tanh(z)
        sech2 = 1.0 - h * h
        dh = sech2 * dz
        d2h = sech2 * d2z - 2.0 * h * sech2 * dz * dz
        res = _residual(y, W.shape[0], W.shape[1])
        if res is not None:
            h = h + res
            dh = dh + _residual(dy, W.shape[0], W.shape[1])
            d2h = d2h + _residual(d2y, W.shape[0], W.shape[1])
        y, dy, d2y = h, dh, d2h
    return y, dy, d2y
