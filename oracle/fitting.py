"""Fitting net: descriptor D_i -> atomic energy E_i, and dE/dD (oracle).

Paper Sec. II: the descriptor is passed to a fully connected network, the
fitting net, which outputs E^i; Sec. III sets its sizes to (240, 240, 240).
Reading (the paper gives only the sizes): with x = D_i flattened row-major
(M x M' values),

    h_1 = tanh(x W_1 + b_1)
    h_l = h_{l-1} + tanh(h_{l-1} W_l + b_l)    l = 2, 3 (equal widths: residual)
    E_i = h_3 . w_out + b_out,

the same residual rule as the embedding net here.  The backward
pass is the chain rule written out layer by layer (delta_l = dE/dh_l):

    delta_3 = w_out
    delta_{l-1} = delta_l + W_l ((1 - t_l^2) * delta_l)   l = 3, 2   (t_l = tanh(.))
    dE/dx = W_1 ((1 - t_1^2) * delta_1).

Test infrastructure: float64 numpy; matrix products are library calls.
"""
import numpy as np


def forward(D, net):
    """E [n] and the tanh outputs t_1..t_3 (each [n, width]) for D [n, M, M']."""
    x = D.reshape(D.shape[0], -1)
    W, b = net["W"], net["b"]
    t = [np.tanh(x @ W[0] + b[0])]
    h = t[0]
    for l in (1, 2):
        t.append(np.tanh(h @ W[l] + b[l]))
        h = h + t[l]
    E = h @ net["w_out"] + net["b_out"]
    return E, t


def backward(D, net):
    """dE_i/dD_i [n, M, M'] (each atom's energy against its own descriptor)."""
    _, t = forward(D, net)
    W = net["W"]
    n = D.shape[0]
    delta = np.broadcast_to(net["w_out"], (n, len(net["w_out"]))).copy()
    for l in (2, 1):
        delta = delta + ((1.0 - t[l] ** 2) * delta) @ W[l].T
    dx = ((1.0 - t[0] ** 2) * delta) @ W[0].T
    return dx.reshape(D.shape)
