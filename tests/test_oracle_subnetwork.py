"""Pins of the oracle's memory subnetwork (Sec. 3.1): it reduces to the pinned
activation layer when the dense parts are identities, and its gradients match
directional finite differences of an independent fp64 evaluation with the
neighbour selection held fixed.
"""
import numpy as np

import oracle
from oracle import subnetwork as sub

K = (4, 6, 4, 6, 4, 6, 4, 6)


def _params(w, rng, scale=1.0):
    m = 64
    return {
        "W1": rng.standard_normal((w, w)) * scale / np.sqrt(w), "b1": rng.standard_normal(w) * 0.1,
        "mu": rng.standard_normal(w) * 0.1, "var": rng.uniform(0.5, 2.0, w), "eps": 1e-5,
        "gamma": rng.uniform(0.5, 1.5, w), "beta": rng.standard_normal(w) * 0.1,
        "W2": rng.standard_normal((w, w // 16 * m)) / np.sqrt(w // 16 * m), "b2": rng.standard_normal(w) * 0.1,
    }


def test_identity_dense_parts_reduce_to_theta():
    rng = np.random.default_rng(1)
    w, T = 32, 50
    table = rng.standard_normal((int(np.prod(K)), 64))
    p = {"W1": np.eye(w), "b1": np.zeros(w), "mu": np.zeros(w), "var": np.ones(w), "eps": 0.0,
         "gamma": np.ones(w), "beta": np.zeros(w), "W2": np.zeros((w, 128)), "b2": np.zeros(w)}
    p["W2"][:16, :16] = np.eye(16)         # first 16 values of head 0
    p["W2"][16:, 64:80] = np.eye(16)       # first 16 values of head 1
    x = rng.standard_normal((T, w)).astype(np.float32)
    y, _ = sub.forward(x, p, K, table)
    q, s = oracle.theta_coords(x.reshape(T, 2, 16), K)
    nb = oracle.neighbors(q, K)
    th = oracle.theta_forward(nb, oracle.gather_rows(table, nb["slot"]), s)
    np.testing.assert_allclose(y[:, :16], th[:, 0, :16], rtol=1e-13)
    np.testing.assert_allclose(y[:, 16:], th[:, 1, :16], rtol=1e-13)


def _fixed_eval(x, p, table, st):
    """fp64 forward with the lattice points of every lookup fixed (the lists in st)."""
    T, w = x.shape
    h = w // 16
    pre = x @ p["W1"].T + p["b1"]
    z = (((pre - p["mu"]) / np.sqrt(p["var"] + p["eps"])) * p["gamma"] + p["beta"]).reshape(T, h, 16)
    z0 = st["z"]
    c = np.asarray(K, np.float64) / (2 * np.pi)
    a, b = z[..., 0::2], z[..., 1::2]
    x_lat = st["nb"]["x"].astype(np.float64) + 2 * c * (np.arctan2(b, a) - np.arctan2(z0[..., 1::2], z0[..., 0::2]))
    s = 1 / np.sum(1 / np.sqrt(a * a + b * b), axis=-1)
    k = st["nb"]["lift"].astype(np.float64)
    valid = st["nb"]["slot"] >= 0
    d2 = np.sum((x_lat[..., None, :] - k) ** 2, axis=-1)
    wts = np.where(valid, (1 - d2 / 8) ** 4, 0.0)
    rows = table[np.where(valid, st["nb"]["slot"], 0)]
    th = (s[..., None] * np.einsum("thj,thjm->thm", wts, rows)).reshape(T, -1)
    return th @ p["W2"].T + p["b2"]


def test_gradients_match_directional_finite_differences():
    rng = np.random.default_rng(2)
    w, T = 32, 40
    table = rng.standard_normal((int(np.prod(K)), 64))
    p = _params(w, rng, scale=3.0)
    x = rng.standard_normal((T, w))
    y, st = sub.forward(x, p, K, table)
    dy = rng.standard_normal(y.shape)
    g = sub.backward(dy, p, K, table, st)
    # the oracle's forward rounds q to fp32; evaluate the fixed-selection
    # function around the same base point (x_lat from the oracle's lists)
    st["z"] = st["z"].astype(np.float32).astype(np.float64)
    h = 1e-6
    for name in ("x", "W1", "b1", "gamma", "beta", "W2", "b2"):
        for trial in range(3):
            d = rng.standard_normal(x.shape if name == "x" else p[name].shape)
            if name == "x":
                fp = _fixed_eval(x + h * d, p, table, st)
                fm = _fixed_eval(x - h * d, p, table, st)
                an = np.sum(g["x"] * d)
            else:
                pp, pm = dict(p), dict(p)
                pp[name] = p[name] + h * d
                pm[name] = p[name] - h * d
                fp = _fixed_eval(x, pp, table, st)
                fm = _fixed_eval(x, pm, table, st)
                an = np.sum(g[name] * d)
            fd = np.sum(dy * (fp - fm)) / (2 * h)
            np.testing.assert_allclose(an, fd, rtol=2e-5, err_msg=name)
    # table: the slice is linear in it
    uniq, acc = g["table"]
    probe = rng.standard_normal(table.shape)
    tp = table + probe
    yp, _ = sub.forward(x, p, K, tp)
    np.testing.assert_allclose(np.sum(dy * (yp - y)), np.sum(acc * probe[uniq]), rtol=1e-10)
