"""Pins of the oracle's memory subnetwork (Sec. 3.1): it reduces to the pinned
activation layer when the dense parts are identities; in training form the
normalised features have zero batch mean and a batch second moment of
var / (var + eps) (biased variance), the output does not depend on b1 (the
batch mean removes it) and the b1 gradient vanishes; and its gradients match
directional finite differences of an independent fp64 evaluation with the
neighbour selection held fixed, in inference and in training form.
"""
import numpy as np
import pytest

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


def test_training_normalisation_closed_forms():
    rng = np.random.default_rng(3)
    w, T = 32, 48
    table = rng.standard_normal((int(np.prod(K)), 64))
    p = _params(w, rng, scale=3.0)
    x = rng.standard_normal((T, w))
    y, st = sub.forward(x, p, K, table, training=True)
    pre = st["pre"]
    c = pre - pre.sum(0) / T
    var = np.einsum("tw,tw->w", c, c) / T
    np.testing.assert_allclose(st["xhat"].sum(0) / T, 0.0, atol=1e-13)
    np.testing.assert_allclose(np.einsum("tw,tw->w", st["xhat"], st["xhat"]) / T, var / (var + p["eps"]),
                               rtol=1e-12)
    # the batch mean removes any shift of the pre-activations
    p2 = dict(p)
    p2["b1"] = p["b1"] + rng.standard_normal(w)
    y2, _ = sub.forward(x, p2, K, table, training=True)
    np.testing.assert_allclose(y2, y, rtol=1e-9, atol=1e-12)
    g = sub.backward(rng.standard_normal(y.shape), p, K, table, st)
    assert np.abs(g["b1"]).max() <= 1e-10 * np.abs(g["beta"]).max()


def _fixed_eval(x, p, table, st, training=False):
    """fp64 forward with the lattice points of every lookup fixed (the lists in st)."""
    T, w = x.shape
    h = w // 16
    pre = x @ p["W1"].T + p["b1"]
    if training:
        mean = pre.sum(0) / T
        var = ((pre - mean) ** 2).sum(0) / T
    else:
        mean, var = p["mu"], p["var"]
    z = (((pre - mean) / np.sqrt(var + p["eps"])) * p["gamma"] + p["beta"]).reshape(T, h, 16)
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


@pytest.mark.parametrize("training", [False, True])
def test_gradients_match_directional_finite_differences(training):
    rng = np.random.default_rng(2)
    w, T = 32, 40
    table = rng.standard_normal((int(np.prod(K)), 64))
    p = _params(w, rng, scale=3.0)
    x = rng.standard_normal((T, w))
    y, st = sub.forward(x, p, K, table, training=training)
    dy = rng.standard_normal(y.shape)
    g = sub.backward(dy, p, K, table, st)
    # the oracle's forward rounds q to fp32; evaluate the fixed-selection
    # function around the same base point (x_lat from the oracle's lists)
    st["z"] = st["zq"].astype(np.float64)
    h = 1e-6
    for name in ("x", "W1", "b1", "gamma", "beta", "W2", "b2"):
        for trial in range(3):
            d = rng.standard_normal(x.shape if name == "x" else p[name].shape)
            if name == "x":
                fp = _fixed_eval(x + h * d, p, table, st, training)
                fm = _fixed_eval(x - h * d, p, table, st, training)
                an = np.sum(g["x"] * d)
            else:
                pp, pm = dict(p), dict(p)
                pp[name] = p[name] + h * d
                pm[name] = p[name] - h * d
                fp = _fixed_eval(x, pp, table, st, training)
                fm = _fixed_eval(x, pm, table, st, training)
                an = np.sum(g[name] * d)
            fd = np.sum(dy * (fp - fm)) / (2 * h)
            # atol: the b1 derivative vanishes in training form, where the
            # difference quotient is rounding noise (~1e-10)
            np.testing.assert_allclose(an, fd, rtol=2e-5, atol=1e-8, err_msg=name)
    # table: the slice is linear in it
    uniq, acc = g["table"]
    probe = rng.standard_normal(table.shape)
    tp = table + probe
    yp, _ = sub.forward(x, p, K, tp, training=training)
    np.testing.assert_allclose(np.sum(dy * (yp - y)), np.sum(acc * probe[uniq]), rtol=1e-10)
