"""Pins of the oracle's variable-k and untruncated lookups (Sec. 2.2 and 2.5:
the sum over every lattice point in the support; Sec. 2.6: the truncation to
the closest k).

* the whole support against the all-locations brute force on tiny tori;
* the closest k are a prefix of the closest k' > k, and of the whole support;
* total weight of the untruncated kernel: 1 at lattice points and deep holes,
  within [0.85122, 1] everywhere (Sec. 2.5), equal to the oracle's own
  full-support sum;
* fp32 rounding of the distance recipe can admit points at distance exactly
  sqrt 8 (the support is an open ball in exact arithmetic): counts above
  Table 1's 121 occur next to lattice points, but never above 1 + 240.
"""
import numpy as np
import pytest

import oracle
from bruteforce import all_locations, support

FACTS_MIN_TOTAL = 0.85122


@pytest.mark.parametrize("K", [(2,) * 8, (4,) * 8, (2, 4, 2, 4, 4, 2, 4, 2)])
def test_whole_support_matches_bruteforce(K):
    rng = np.random.default_rng(77 + sum(K))
    q = np.concatenate([np.zeros((1, 8)), np.full((1, 8), 0.5), rng.random((30, 8)) * np.asarray(K)]).astype(
        np.float32)
    nb = oracle.neighbors(q, K, k=0)
    locs = all_locations(K)
    for l in range(q.shape[0]):
        d, s, k = support(nb["x"][l], K, locs)
        n = d.size
        assert nb["count"][l] == n
        np.testing.assert_array_equal(nb["slot"][l, :n], s)
        np.testing.assert_array_equal(nb["d2"][l, :n].view(np.uint32), d.view(np.uint32))
        np.testing.assert_array_equal(nb["lift"][l, :n], k)
        assert np.all(nb["slot"][l, n:] == -1)


def test_closest_k_are_prefixes():
    K = (8,) * 8
    q = (np.random.default_rng(5).random((500, 8)) * 8).astype(np.float32)
    full = oracle.neighbors(q, K, k=0)
    for k in (16, 32, 64):
        nb = oracle.neighbors(q, K, k=k)
        np.testing.assert_array_equal(nb["slot"], full["slot"][:, :k])
        np.testing.assert_array_equal(nb["w64"], full["w64"][:, :k])
        assert np.all((nb["slot"] >= 0).sum(1) == np.minimum(full["count"], k))


def test_untruncated_total_weight():
    K = (8,) * 8
    rng = np.random.default_rng(6)
    q = (rng.random((4000, 8)) * 8).astype(np.float32)
    special = np.array([[0] * 8, [1, 0, 0, 0, 0, 0, 0, 0], [0.5] * 8], np.float32)  # point, deep hole, odd point
    nb = oracle.neighbors(np.concatenate([special, q]), K, k=0)
    tot = nb["w64"].sum(1)
    np.testing.assert_allclose(tot, nb["wsum"], rtol=1e-14)
    np.testing.assert_allclose(tot[:3], 1.0, rtol=1e-15)
    assert tot.min() >= FACTS_MIN_TOTAL and tot.max() <= 1.0 + 1e-15
    # a constant table reads back the total weight through the untruncated sum
    ones = np.ones((int(np.prod(K)), 3))
    phi = oracle.forward(nb, oracle.gather_rows(ones, nb["slot"]))
    np.testing.assert_allclose(phi[:, 0], tot, rtol=1e-14)


def test_rounding_can_admit_the_shell_but_never_beyond_it():
    """x = t (1,...,1) next to the origin: the 126 shell points orthogonal to
    (1,...,1) sit at r^2 = 8 + 8 t^2 exactly; the recipe can round some of them
    below 8.  The closed ball of radius sqrt 8 around a lattice point holds
    1 + 240 points, the most any ball of that radius holds."""
    K = (8,) * 8
    ts = np.float32(3.801106e-08) * np.arange(1, 200, dtype=np.float32)
    q = np.repeat(ts[:, None], 8, axis=1).astype(np.float32)
    nb = oracle.neighbors(q, K, k=0)
    assert nb["count"].max() > 121
    assert nb["count"].max() <= 241
    # the admitted extra points are exactly at distance sqrt 8 in exact arithmetic
    for l in np.nonzero(nb["count"] > 121)[0][:5]:
        n = nb["count"][l]
        assert np.all(nb["slot"][l, :n] >= 0) and np.all(nb["slot"][l, n:] == -1)  # every point listed
        assert np.all(nb["d64"][l, :n] < 8 + 1e-5)
