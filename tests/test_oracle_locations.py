"""The location map Lambda -> [0, N) of the oracle (Sec. 2.2: M = Lambda / L_K).

Pinned by the two properties that define a labelling of the quotient: it is
constant on cosets of L_K (torus periods 2K_i e_i at the Lambda scale) and it is
a bijection from the N cosets onto [0, N).
"""
import itertools

import numpy as np
import pytest

import oracle


def _coset_reps(K):
    """One representative per coset of L_K in Lambda, listed without any index formula."""
    reps = []
    ranges = [range(2 * k) for k in K]
    for k in itertools.product(*ranges):
        k = np.array(k)
        if len(set(k % 2)) == 1 and k.sum() % 4 == 0:
            reps.append(k)
    return np.array(reps, np.int32)


@pytest.mark.parametrize("K", [(2,) * 8, (2, 4, 2, 2, 4, 2, 2, 2), (4, 2, 2, 6, 2, 2, 2, 2)])
def test_location_is_bijection(K):
    reps = _coset_reps(K)
    N = int(np.prod(K))
    assert reps.shape[0] == N  # |Lambda / L_K| = prod(2K_i) / det(Lambda) = prod K_i
    loc = oracle.locations(reps, K)
    assert loc.min() == 0 and loc.max() == N - 1
    assert np.unique(loc).size == N


@pytest.mark.parametrize("K", [(2,) * 8, (4, 6, 8, 2, 4, 10, 2, 4)])
def test_location_is_periodic(K):
    rng = np.random.default_rng(31)
    eps = rng.integers(0, 2, size=500)
    k = 2 * rng.integers(-20, 20, size=(500, 8)) + eps[:, None]
    bad = (k.sum(1) % 4) != 0
    k[bad, 0] += 2  # fix the sum (keeps the parity class)
    assert np.all(k.sum(1) % 4 == 0)
    base = oracle.locations(k, K)
    for i in range(8):
        for n in (-3, 1, 2):
            k2 = k.copy()
            k2[:, i] += 2 * K[i] * n
            np.testing.assert_array_equal(oracle.locations(k2, K), base)
