"""Symmetry properties of the oracle (Sec. 2.4 and Sec. 2.6).

Queries sit on a dyadic grid (multiples of 2^-8 at the Lambda scale), where every
operation of the fp32 distance recipe is exact, so the comparisons are bit-exact.
"""
import numpy as np

import oracle

K8 = (8,) * 8


def _dyadic(rng, n, K):
    x = rng.integers(0, 2 * 256 * np.asarray(K), size=(n, 8)) / 256.0  # Lambda scale in [0,2K)
    return (x / 2).astype(np.float32)


def _sorted_d(nb):
    d = np.where(nb["slot"] >= 0, nb["d2"], np.inf)
    return np.sort(d, axis=-1)


def test_torus_period_leaves_everything_unchanged():
    """Adding a torus period K_i e_i (user scale) changes nothing (Sec. 2.2)."""
    rng = np.random.default_rng(11)
    K = (4, 6, 8, 4, 10, 4, 2, 4)
    q = _dyadic(rng, 64, K)
    base = oracle.neighbors(q, K)
    for i in range(8):
        for sgn in (-1, 1):
            q2 = q.copy()
            q2[:, i] += sgn * K[i]
            nb = oracle.neighbors(q2, K)
            np.testing.assert_array_equal(nb["slot"], base["slot"])
            np.testing.assert_array_equal(nb["d2"].view(np.uint32), base["d2"].view(np.uint32))


def test_lattice_translation_shifts_lifts():
    """Translating by t in Lambda shifts every neighbour lift by t; distances and
    weights are unchanged and locations follow the shifted points."""
    rng = np.random.default_rng(12)
    q = _dyadic(rng, 64, K8)
    base = oracle.neighbors(q, K8)
    for t in ([2, 2, 0, 0, 0, 0, 0, 0], [1, 1, 1, 1, 1, 1, 1, 1], [4, -2, 0, 2, 0, 0, 0, 0],
              [3, 1, 1, 1, 1, 1, -1, 1]):
        t = np.array(t)
        assert t.sum() % 4 == 0 and len(set(t % 2)) == 1
        q2 = q + (t / 2).astype(np.float32)
        nb = oracle.neighbors(q2, K8)
        np.testing.assert_array_equal(_sorted_d(nb).view(np.uint32), _sorted_d(base).view(np.uint32))
        # lifts strictly inside the last kept distance are unique and must shift by t
        # (up to the torus period 2K = 16, as the translated query may wrap);
        # points tied with the 32nd distance are chosen by location, which the
        # translation relabels (their distances are compared above)
        for l in range(q.shape[0]):
            okb = base["slot"][l] >= 0
            okn = nb["slot"][l] >= 0
            last = base["d2"][l][okb].max()
            a = {tuple(v) for v in (base["lift"][l][okb & (base["d2"][l] < last)] + t) % 16}
            b = {tuple(v) for v in nb["lift"][l][okn & (nb["d2"][l] < last)] % 16}
            assert a == b


def _weyl_images(x, rng):
    """A few elements of W(E8) applied to Lambda-scale points x[n,8]:
    coordinate permutations, even sign changes and the reflection in the root
    (1,...,1) -- the last one lies outside the signed-permutation subgroup
    used by the fast search (Sec. 2.6: index 135)."""
    outs = []
    outs.append(x[:, rng.permutation(8)])
    s = np.where(rng.random(8) < 0.5, -1.0, 1.0)
    if (s < 0).sum() % 2:
        s[0] = -s[0]
    outs.append(x * s)
    r = np.ones(8)
    outs.append(x - (x @ r / 4.0)[:, None] * r[None, :])
    return outs


def test_support_distances_invariant_under_e8_reflections():
    """The multiset of distances to Lambda is invariant under the isometries of
    Lambda, including the reflection outside W(D8) (Sec. 2.4, 2.6)."""
    rng = np.random.default_rng(13)
    K = (12,) * 8
    x = rng.integers(-256 * 16, 256 * 16, size=(48, 8)) / 256.0
    base = oracle.neighbors((np.mod(x, 24) / 2).astype(np.float32), K)
    for xi in _weyl_images(x, rng):
        nb = oracle.neighbors((np.mod(xi, 24) / 2).astype(np.float32), K)
        np.testing.assert_array_equal(nb["count"], base["count"])
        np.testing.assert_array_equal(_sorted_d(nb).view(np.uint32), _sorted_d(base).view(np.uint32))
        np.testing.assert_array_equal(nb["wsum"], base["wsum"])


def test_index_135():
    """Sec. 2.6: |W(E8)| / (8! * 2^7) = 135."""
    import math
    order_we8 = 696729600  # 2^14 3^5 5^2 7
    assert order_we8 == 2 ** 14 * 3 ** 5 * 5 ** 2 * 7
    assert order_we8 // (math.factorial(8) * 2 ** 7) == 135
