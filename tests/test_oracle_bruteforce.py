"""Oracle vs the all-locations brute force on tiny tori (K = 2, 4, mixed).

Pins the oracle's enumeration, distance recipe, support test and ordering
(Sec. 2.2, 2.5, 2.6) against an independent enumeration of every location of
the torus and every lift of it.
"""
import numpy as np
import pytest

import oracle
from bruteforce import all_locations, support

TORI = [(2,) * 8, (4,) * 8, (2, 4, 2, 4, 4, 2, 4, 2), (6, 2, 2, 4, 2, 2, 2, 2)]


def _queries(K, n, rng):
    K = np.asarray(K, np.float32)
    q = (rng.random((n, 8)) * K).astype(np.float32)
    # out-of-range and negative coordinates exercise the fmod wrap
    q[: n // 8] -= (K * rng.integers(-2, 3, size=(n // 8, 8))).astype(np.float32)
    return q


def _special(K):
    Kf = np.asarray(K, np.float32)
    pts = [
        np.zeros(8),                              # lattice point
        np.array([1, 0, 0, 0, 0, 0, 0, 0.0]),     # deep hole (x = (2,0,..,0))
        np.full(8, 0.5),                          # odd-coset lattice point
        np.array([0.5, 0.5, 0, 0, 0, 0, 0, 0]),   # hole-like point
        np.array([0.25, 0.125, 0.0625, 0, 0.5, 0.75, 0.375, 0.875]),  # dyadic
        np.array([1, 1, 0, 0, 0, 0, 0, 0.0]) + 2.0 ** -9,
    ]
    out = [np.mod(p, Kf).astype(np.float32) for p in pts]
    return np.stack(out)


@pytest.mark.parametrize("K", TORI)
def test_oracle_matches_bruteforce(K):
    rng = np.random.default_rng(1234 + sum(K))
    q = np.concatenate([_special(K), _queries(K, 40, rng)])
    nb = oracle.neighbors(q, K)
    locs = all_locations(K)
    for l in range(q.shape[0]):
        d, s, k = support(nb["x"][l], K, locs)
        assert nb["count"][l] == d.size, (l, nb["count"][l], d.size)
        n = min(32, d.size)
        np.testing.assert_array_equal(nb["slot"][l, :n], s[:n])
        np.testing.assert_array_equal(nb["d2"][l, :n].view(np.uint32), d[:n].view(np.uint32))
        np.testing.assert_array_equal(nb["lift"][l, :n], k[:n])
        assert np.all(nb["slot"][l, n:] == -1)
        assert np.all(nb["w64"][l, n:] == 0)


def test_bruteforce_x_is_exact_fmod():
    rng = np.random.default_rng(7)
    K = (4,) * 8
    q = _queries(K, 64, rng)
    nb = oracle.neighbors(q, K)
    x = np.fmod(np.float32(2) * q, np.float32(8)).astype(np.float32)
    np.testing.assert_array_equal(nb["x"].view(np.uint32), x.view(np.uint32))


def test_k2_has_repeated_locations():
    """At K = 2 the torus side (4) is shorter than the support diameter (2*sqrt 8),
    so one location can be reached through two lifts (lift semantics)."""
    rng = np.random.default_rng(3)
    K = (2,) * 8
    q = _queries(K, 200, rng)
    nb = oracle.neighbors(q, K)
    rep = 0
    for l in range(q.shape[0]):
        s = nb["slot"][l][nb["slot"][l] >= 0]
        rep += int(np.unique(s).size < s.size)
    assert rep > 0
