"""Memory-augmented subnetwork of Sec. 3.1 in fp64 -- TEST INFRASTRUCTURE ONLY
(imported by the tests only; the product never imports it).

y = W2 theta(BN(W1 x + b1)) + b2, with
  * W1: R^w -> R^w (dense affine), BN: batch normalisation of the query
    vector (Sec. 4.1 uses it for the LRAM queries), here in inference form
    (running mean mu, running variance var, eps, scale gamma, shift beta);
  * theta: the activation layer of Sec. 2.3 with (n, m, h) = (8, 64, w/16):
    the w query features are h heads of 8 complex numbers (16 reals,
    interleaved), each head's lookup returns m = 64 values, h*m = 4w;
  * W2: R^{4w} -> R^w (dense affine).
The dense parts are plain matrix products; theta is the oracle's own
(``oracle.theta_*``).  The backward follows the chain rule through each of
these steps with the neighbour selection held fixed.
"""
from __future__ import annotations

import numpy as np

from . import gather_rows, neighbors, theta_coords, theta_forward, theta_grad_table_rows, theta_grad_z


def forward(x, p, K, table):
    """x [T, w]; p: dict of fp64 arrays W1 [w, w], b1, mu, var, gamma, beta, W2 [w, 4w], b2, eps.
    Returns y [T, w] and the saved state for backward."""
    x = np.asarray(x, np.float64)
    T, w = x.shape
    h = w // 16
    pre = x @ p["W1"].T + p["b1"]
    inv = 1.0 / np.sqrt(p["var"] + p["eps"])
    zf = (pre - p["mu"]) * inv * p["gamma"] + p["beta"]
    z = zf.reshape(T, h, 16)
    q, s = theta_coords(z.astype(np.float32), K)
    nb = neighbors(q, K)
    rows = gather_rows(table, nb["slot"])
    th = theta_forward(nb, rows, s).reshape(T, h * table.shape[1])
    y = th @ p["W2"].T + p["b2"]
    return y, dict(x=x, z=z, th=th, q=q, s=s, nb=nb, rows=rows, inv=inv, pre=pre)


def backward(dy, p, K, table, st, table_weights: str = "w64"):
    """Gradients of <dy, y> with respect to x, W1, b1, gamma, beta, W2, b2 and
    the table (as (unique rows, rows), with the kernel weights ``table_weights``
    as in ``oracle.grad_table_rows``); fp64."""
    dy = np.asarray(dy, np.float64)
    T, w = dy.shape
    h = w // 16
    m = table.shape[1]
    g = {"W2": dy.T @ st["th"], "b2": dy.sum(0)}
    dth = (dy @ p["W2"]).reshape(T, h, m)
    dz = theta_grad_z(st["z"].astype(np.float32), K, st["nb"], st["rows"], st["s"], dth).reshape(T, w)
    g["table"] = theta_grad_table_rows(st["nb"], st["s"], dth, table_weights)
    norm = (st["pre"] - p["mu"]) * st["inv"]
    g["gamma"] = (dz * norm).sum(0)
    g["beta"] = dz.sum(0)
    dpre = dz * p["gamma"] * st["inv"]
    g["W1"] = dpre.T @ st["x"]
    g["b1"] = dpre.sum(0)
    g["x"] = dpre @ p["W1"]
    return g
