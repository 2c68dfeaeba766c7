"""Memory-augmented subnetwork of Sec. 3.1 in fp64 -- TEST INFRASTRUCTURE ONLY
(imported by the tests only; the product never imports it).

y = W2 theta(BN(W1 x + b1)) + b2, with
  * W1: R^w -> R^w (dense affine), BN: batch normalisation of the query
    vector (Sec. 4.1 uses it for the LRAM queries) with eps, scale gamma and
    shift beta, in inference form (running mean mu and variance var) or in
    training form (the mean and the biased variance of the batch's T rows,
    through which the gradient of every row then also flows);
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


def _normalise(pre, p, training):
    """(pre - mean) / sqrt(var + eps) per feature, the mean and the inverse
    deviation: the batch's statistics (biased variance) when training, the
    running ones p["mu"], p["var"] otherwise."""
    if training:
        mu = pre.mean(0)
        var = ((pre - mu) ** 2).mean(0)
    else:
        mu, var = p["mu"], p["var"]
    inv = 1.0 / np.sqrt(var + p["eps"])
    return (pre - mu) * inv, mu, inv


def forward(x, p, K, table, training=False, queries=None):
    """x [T, w]; p: dict of fp64 arrays W1 [w, w], b1, mu, var, gamma, beta, W2 [w, 4w], b2, eps.
    training: batch-statistics normalisation.  queries: the fp32 activation
    inputs z [T, w] the lookups take (default: the fp64 z rounded to fp32).
    Returns y [T, w] and the saved state for backward."""
    x = np.asarray(x, np.float64)
    T, w = x.shape
    h = w // 16
    pre = x @ p["W1"].T + p["b1"]
    xhat, mu, inv = _normalise(pre, p, training)
    zf = xhat * p["gamma"] + p["beta"]
    z = zf.reshape(T, h, 16)
    zq = z.astype(np.float32) if queries is None else np.asarray(queries, np.float32).reshape(T, h, 16)
    q, s = theta_coords(zq, K)
    nb = neighbors(q, K)
    rows = gather_rows(table, nb["slot"])
    th = theta_forward(nb, rows, s).reshape(T, h * table.shape[1])
    y = th @ p["W2"].T + p["b2"]
    return y, dict(x=x, z=z, zq=zq, th=th, q=q, s=s, nb=nb, rows=rows, inv=inv, mu=mu, xhat=xhat, pre=pre,
                   training=training)


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
    dz = theta_grad_z(st["zq"], K, st["nb"], st["rows"], st["s"], dth).reshape(T, w)
    g["table"] = theta_grad_table_rows(st["nb"], st["s"], dth, table_weights)
    g["gamma"] = (dz * st["xhat"]).sum(0)
    g["beta"] = dz.sum(0)
    dxhat = dz * p["gamma"]
    if st["training"]:
        # the batch mean and variance depend on every row
        dpre = st["inv"] * (dxhat - dxhat.mean(0) - st["xhat"] * (dxhat * st["xhat"]).mean(0))
    else:
        dpre = dxhat * st["inv"]
    g["W1"] = dpre.T @ st["x"]
    g["b1"] = dpre.sum(0)
    g["x"] = dpre @ p["W1"]
    return g
