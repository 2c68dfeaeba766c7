"""Pins of the oracle's activation layer (Sec. 2.3) against facts that do not
come from the oracle's own formulas: closed forms at quarter turns (where the
torus coordinate lands on a lattice point, so phi is one table row), the scale
of the displayed formula, the homogeneity the section states, finite
differences of an independent fp64 evaluation, and the adjoint identity for
the value table.
"""
import numpy as np
import pytest

import oracle

K4 = (4,) * 8


def _table(N, m, seed=0):
    return np.random.default_rng(seed).standard_normal((N, m))


def _theta(z, K, table):
    q, s = oracle.theta_coords(z, K)
    nb = oracle.neighbors(q, K)
    rows = oracle.gather_rows(table, nb["slot"])
    return oracle.theta_forward(nb, rows, s), q, s, nb, rows


def _unit(re, im):
    z = np.zeros((1, 16), np.float32)
    z[0, 0::2] = re
    z[0, 1::2] = im
    return z


@pytest.mark.parametrize("re,im,point", [(1, 0, 0), (0, 1, 2), (-1, 0, 4), (0, -1, -2)])
def test_quarter_turns_hit_lattice_points(re, im, point):
    """arg z = 0, pi/2, pi, -pi/2 give torus coordinate 0, K/4, K/2, -K/4; at
    K = 4 that is the Lambda-scale point (2q, ..., 2q), a lattice point of
    2*E8, so phi is exactly its row and theta is that row times 1/8."""
    table = _table(4 ** 8, 5)
    th, q, s, nb, _ = _theta(_unit(re, im), K4, table)
    assert np.all(q == np.float32(point / 2))
    assert s[0] == 0.125
    assert nb["count"][0] == 1 and nb["w64"][0, 0] == 1.0
    loc = oracle.locations(np.full((1, 8), point, np.int32), K4)[0]
    np.testing.assert_array_equal(th[0], table[loc] / 8)


def test_origin_row_is_row_zero():
    """The origin is location 0 of the bijection (eps = 0, Y = 0)."""
    table = _table(4 ** 8, 3)
    th, *_ = _theta(_unit(1, 0), K4, table)
    np.testing.assert_array_equal(th[0], table[0] / 8)


def test_scale_is_reciprocal_sum_of_reciprocal_moduli():
    """The displayed formula: s = (sum 1/|z_i|)^-1 (not the harmonic mean n/sum)."""
    r = np.array([1, 2, 4, 8, 1, 2, 4, 8], np.float32)
    table = _table(4 ** 8, 3)
    th, q, s, *_ = _theta(_unit(r, 0), K4, table)
    assert s[0] == 1 / 3.75
    np.testing.assert_allclose(th[0], table[0] / 3.75, rtol=1e-15)
    # the same moduli at any phases: s depends on |z| only
    rng = np.random.default_rng(3)
    ph = rng.random(8) * 2 * np.pi
    _, s2 = oracle.theta_coords(_unit(r * np.cos(ph), r * np.sin(ph)), K4)
    np.testing.assert_allclose(s2[0], 1 / 3.75, rtol=1e-6)


def test_zero_and_nonfinite_entries():
    table = _table(4 ** 8, 3)
    z = np.random.default_rng(4).standard_normal((3, 16)).astype(np.float32)
    z[0, 4:6] = 0.0          # z_2 = 0: scale 0, output 0 (the continuous extension)
    z[1, 7] = np.inf
    z[2, 0] = np.nan
    th, q, s, nb, rows = _theta(z, K4, table)
    assert np.all(s == 0) and np.all(th == 0)
    G = np.ones((3, 3))
    assert np.all(oracle.theta_grad_z(z, K4, nb, rows, s, G) == 0)
    assert np.all(nb["count"][1:] == 0)


def test_homogeneous_of_degree_one():
    """Sec. 2.3: theta(lambda z) = lambda theta(z) for lambda >= 0 (exact for
    powers of two, where arg and the moduli scale without rounding)."""
    K = (4, 6, 8, 4, 6, 8, 4, 6)
    table = _table(int(np.prod(K)), 4, seed=5)
    z = np.random.default_rng(6).standard_normal((64, 16)).astype(np.float32)
    th, *_ = _theta(z, K, table)
    for lam in (0.25, 8.0, 2.0 ** 20):
        th2, *_ = _theta((z * np.float32(lam)).astype(np.float32), K, table)
        np.testing.assert_allclose(th2, lam * th, rtol=1e-14, atol=0)
    th0, *_ = _theta(np.zeros_like(z), K, table)
    assert np.all(th0 == 0)


def _theta_fixed(z64, K, nb, table, x0, t0):
    """Independent fp64 evaluation of theta with the selection held fixed:
    the Lambda-scale point moves by 2 c (arg z - arg z0) from the base x0."""
    c = np.asarray(K, np.float64) / (2 * np.pi)
    a, b = z64[0::2], z64[1::2]
    x = x0 + 2 * c * (np.arctan2(b, a) - t0)
    s = 1 / np.sum(1 / np.sqrt(a * a + b * b))
    k = nb["lift"].astype(np.float64)
    valid = nb["slot"] >= 0
    d2 = np.sum((x[None, :] - k) ** 2, axis=1)
    w = np.where(valid, (1 - d2 / 8) ** 4, 0.0)
    rows = table[np.where(valid, nb["slot"], 0)]
    return s * (w @ rows)


def test_grad_z_matches_finite_differences():
    K = (4, 6, 8, 4, 6, 8, 4, 6)
    m = 3
    table = _table(int(np.prod(K)), m, seed=7)
    rng = np.random.default_rng(8)
    z = (rng.standard_normal((40, 16)) * rng.uniform(0.3, 3.0, (40, 1))).astype(np.float32)
    G = rng.standard_normal((40, m))
    th, q, s, nb, rows = _theta(z, K, table)
    gz = oracle.theta_grad_z(z, K, nb, rows, s, G)
    h = 1e-6
    checked = 0
    for l in range(z.shape[0]):
        nbl = {k: v[l] for k, v in nb.items()}
        # skip lookups with a neighbour within 1e-4 of the support edge
        if np.any((nbl["slot"] >= 0) & (nbl["d64"] > 8 - 1e-4)):
            continue
        z64 = z[l].astype(np.float64)
        t0 = np.arctan2(z64[1::2], z64[0::2])
        x0 = nbl["x"].astype(np.float64)
        fd = np.empty(16)
        for i in range(16):
            e = np.zeros(16)
            e[i] = h
            fp = _theta_fixed(z64 + e, K, nbl, table, x0, t0) @ G[l]
            fm = _theta_fixed(z64 - e, K, nbl, table, x0, t0) @ G[l]
            fd[i] = (fp - fm) / (2 * h)
        np.testing.assert_allclose(gz[l], fd, rtol=2e-5, atol=1e-7 * np.abs(fd).max())
        checked += 1
    assert checked >= 30


def test_grad_table_adjoint():
    """<G, theta with table dV_probe> = <dV(G), dV_probe> (theta is linear in the table)."""
    K = (2, 4, 6, 8, 2, 4, 6, 8)
    N = int(np.prod(K))
    m = 2
    rng = np.random.default_rng(9)
    z = rng.standard_normal((300, 16)).astype(np.float32)
    G = rng.standard_normal((300, m))
    probe = rng.standard_normal((N, m))
    q, s = oracle.theta_coords(z, K)
    nb = oracle.neighbors(q, K)
    lhs = np.sum(G * oracle.theta_forward(nb, oracle.gather_rows(probe, nb["slot"]), s))
    uniq, acc = oracle.theta_grad_table_rows(nb, s, G)
    rhs = np.sum(acc * probe[uniq])
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12)
