"""CPU model of the GPU neighbour search, checked against the oracle.

The GPU kernels do not enumerate lattice points; they follow Sec. 2.6: find the
closest lattice point c, carry x - c into the fundamental region F by a signed
permutation (even number of sign changes), scan the fixed candidate list of
points near F (``csrc/e8_candidates.inc``) mapped back by the inverse isometry,
and keep the closest 32.  This numpy model of that design (written for the
tests, sharing no code with the kernels) must reproduce the oracle's lists
exactly; it validates the candidate table and the reduction on the CPU.
"""
import os
import re
from fractions import Fraction

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INC = os.path.join(ROOT, "paper_2107_03474_amd", "csrc", "e8_candidates.inc")


def _read_lists():
    txt = open(INC).read()
    out = {}
    for name in ("E8_STRICT_INIT", "E8_BOUNDARY_INIT"):
        body = txt[txt.index("#define " + name):]
        body = body[: body.index("}\n") + 1]
        rows = re.findall(r"\{([-\d,\s]+)\}", body)
        out[name] = np.array([[int(v) for v in r.split(",")] for r in rows], np.int64)
    return out["E8_STRICT_INIT"], out["E8_BOUNDARY_INIT"]


STRICT, BOUNDARY = _read_lists()


def _read_fast(suffix=""):
    txt = open(INC).read()
    n = int(re.search(r"#define E8_FAST%s (\d+)" % suffix, txt).group(1))
    bound = float(re.search(r"#define E8_FAST%s_BOUND ([\d.]+)f" % suffix, txt).group(1))
    return n, bound


FAST, FAST_BOUND = _read_fast()
FAST_LIMIT = np.float32(FAST_BOUND - 2.0 ** -7)   # the kernels' margin
FAST2, FAST2_BOUND = _read_fast("2")              # the first tier
FAST2_LIMIT = np.float32(FAST2_BOUND - 2.0 ** -7)


def _d8_round(y):
    r = np.rint(y)
    bad = (r.sum(1) % 2) != 0
    worst = np.argmax(np.abs(y - r), axis=1)
    idx = np.arange(y.shape[0])
    step = np.where(y[idx, worst] > r[idx, worst], 1.0, -1.0)
    r[idx[bad], worst[bad]] += step[bad]
    return r


def _reduce(x):
    """closest point c, F-position r_i of each coordinate and sign s'_i."""
    c0 = 2 * _d8_round(x * np.float32(0.5))
    c1 = 2 * _d8_round((x - np.float32(1)) * np.float32(0.5)) + 1
    d0 = ((x - c0) ** 2).sum(1)
    d1 = ((x - c1) ** 2).sum(1)
    c = np.where((d1 < d0)[:, None], c1, c0).astype(np.int64)
    y = x - c.astype(np.float32)
    a = np.abs(y)
    n = x.shape[0]
    r = np.zeros((n, 8), np.int64)
    for i in range(8):
        for j in range(8):
            if j != i:
                r[:, i] += (a[:, j] > a[:, i]) | ((a[:, j] == a[:, i]) & (j < i))
    neg = y < 0
    odd = neg.sum(1) % 2 == 1
    last = r == 7
    neg = np.where(odd[:, None] & last, ~neg, neg)
    s = np.where(neg, -1, 1)
    return c, r, s


def _recipe(x, k):
    e = x[:, None, :] - k.astype(np.float32)
    sq = e * e
    d = sq[..., 0].copy()
    for i in range(1, 8):
        d = d + sq[..., i]
    return d


def model_neighbors(q, K, fast=False, tiers=None):
    """fast: first the FAST2 candidates nearest to F, then the FAST nearest;
    a set's closest 32 stand when the 32nd is below the bound every later
    candidate respects.  Returns also the number of lookups that needed the
    full scan and the number served by the first tier.  tiers: (count,
    limit) pairs in place of the table's (a test plants a wrong bound there)."""
    K = np.asarray(K)
    x = np.fmod(np.float32(2) * q, (2 * K).astype(np.float32)).astype(np.float32)
    c, r, s = _reduce(x)
    # candidates in original coordinates: k_i = c_i + s_i * p_{r_i}
    def lift(P):
        pr = P[:, r]                    # [ncand, n, 8]: p_{r_i}
        pr = np.transpose(pr, (1, 0, 2))
        return c[:, None, :] + s[:, None, :] * pr
    kS = lift(STRICT)
    dS = _recipe(x, kS)
    out_slots = np.full((q.shape[0], 32), -1, np.int64)
    suspects = 0
    fallbacks = 0
    first_tier = 0
    for l in range(q.shape[0]):
        d, k = dS[l], kS[l]
        if fast:
            for n_set, limit in (tiers or ((FAST2, FAST2_LIMIT), (FAST, FAST_LIMIT))):
                dF = np.sort(d[:n_set])
                if dF.size >= 32 and dF[31] < limit:
                    first_tier += n_set == FAST2
                    d, k = d[:n_set], k[:n_set]
                    break
            else:
                fallbacks += 1
        keep = d < np.float32(8)
        n8 = keep.sum()
        dd = np.sort(d[keep])
        suspect = n8 <= 32 or dd[31] >= np.float32(7.999)
        if suspect:
            suspects += 1
            kB = c[l] + s[l] * BOUNDARY[:, r[l]]
            dB = _recipe(x[l:l + 1], kB[None])[0]
            d = np.concatenate([d, dB])
            k = np.concatenate([k, kB])
            keep = d < np.float32(8)
        d, k = d[keep], k[keep]
        slot = oracle.locations(k.astype(np.int32), K).astype(np.int64)
        bits = d.view(np.uint32).astype(np.int64)
        order = np.lexsort(tuple(k[:, i] for i in range(7, -1, -1)) + (slot, bits))[:32]
        out_slots[l, :order.size] = slot[order]
    if fast:
        return out_slots, suspects, fallbacks, first_tier
    return out_slots, suspects


def test_candidate_table_shape():
    """Sec. 2.6: exactly 232 lattice points lie within sqrt 8 of F."""
    assert STRICT.shape == (232, 8)
    norms = (STRICT ** 2).sum(1)
    assert sorted(np.unique(norms)) == [0, 8, 16]
    assert [(norms == v).sum() for v in (0, 8, 16)] == [1, 149, 82]
    for P in (STRICT, BOUNDARY):
        assert np.all(P.sum(1) % 4 == 0)
        assert np.all((P % 2 == 0).all(1) | (P % 2 == 1).all(1))
    assert len({tuple(v) for v in np.concatenate([STRICT, BOUNDARY])}) == 232 + BOUNDARY.shape[0]


def test_generator_reproduces_committed_table():
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "gen", os.path.join(ROOT, "paper_2107_03474_amd", "csrc", "gen_e8_candidates.py"))
    gen = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(gen)
    info = gen.main(write=False)
    np.testing.assert_array_equal(info["strict"], STRICT)
    np.testing.assert_array_equal(info["boundary"], BOUNDARY)
    assert info["gap"] > 0.5


@pytest.mark.parametrize("K", [(4,) * 8, (8,) * 8, (14,) * 8, (2, 4, 6, 8, 2, 4, 6, 8), (2,) * 8])
def test_model_matches_oracle(K):
    rng = np.random.default_rng(99)
    n = 1500
    q = (rng.random((n, 8)) * np.asarray(K)).astype(np.float32)
    q[:100] -= np.asarray(K, np.float32) * 3          # far outside: exercises the wrap
    slots, _ = model_neighbors(q, K)
    nb = oracle.neighbors(q, K)
    np.testing.assert_array_equal(slots, nb["slot"])


def test_model_special_points():
    K = (8,) * 8
    rho = np.array([0, 1, 2, 3, 4, 5, 6, 23], np.float32)
    pts = [np.zeros(8), np.full(8, 0.5), [1, 0, 0, 0, 0, 0, 0, 0], [0.5] * 7 + [-0.5],
           2.0 ** -11 * rho, np.full(8, 0.5) + 2.0 ** -11 * rho, [1, 1, 0, 0, 0, 0, 0, 0.0],
           [0.25, 0.25, 0.25, 0.25, 0, 0, 0, 0], [0.5, 0.5, 0.5, 0.5, 0.5, 0.5, 0.5, 1.0]]
    q = np.mod(np.array(pts, np.float64), 8).astype(np.float32)
    slots, suspects = model_neighbors(q, K)
    nb = oracle.neighbors(q, K)
    np.testing.assert_array_equal(slots, nb["slot"])
    assert suspects >= 3


def test_fast_set_bound_is_exact():
    """Every strict candidate after the first E8_FAST lies at least
    E8_FAST_BOUND from F (exact distances from the generator's quadratic
    programs), and the first E8_FAST are the nearest to F; likewise the first
    E8_FAST2 and E8_FAST2_BOUND (48/7)."""
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "gen", os.path.join(ROOT, "paper_2107_03474_amd", "csrc", "gen_e8_candidates.py"))
    gen = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(gen)
    d2, sets = gen.project_all(STRICT)
    exact = [gen.exact_dist2(STRICT[i], sets[i]) for i in range(STRICT.shape[0])]
    assert FAST == 192 and FAST % 64 == 0 and FAST2 == 128 and FAST2 % 64 == 0
    assert min(exact[FAST:]) >= FAST_BOUND and max(exact[:FAST]) <= min(exact[FAST:])
    assert min(exact[FAST2:]) == Fraction(48, 7) and max(exact[:FAST2]) <= min(exact[FAST2:])
    assert abs(FAST2_BOUND - 48 / 7) < 1e-7
    assert all(exact[i] <= exact[i + 1] for i in range(len(exact) - 1))


@pytest.mark.parametrize("K", [(4,) * 8, (14,) * 8, (2, 4, 6, 8, 2, 4, 6, 8)])
def test_fast_set_model_matches_oracle(K):
    """The fast-set rule of the kernels' search gives the oracle's lists, on
    random, clustered, dyadic and special queries; the full scan is needed for
    a small share only."""
    rng = np.random.default_rng(123)
    n = 3000
    Kf = np.asarray(K, np.float64)
    q = rng.random((n, 8)) * Kf
    q[:500] = np.mod(np.floor(q[:500] * 16) / 16, Kf)        # dyadic grid: exact ties
    q[500:600] = np.floor(q[500:600])                       # lattice points and deep holes
    q[600:700] = np.floor(q[600:700]) + 1e-6 * rng.standard_normal((100, 8))
    q = q.astype(np.float32)
    got, _, fallbacks, first_tier = model_neighbors(q, K, fast=True)
    nb = oracle.neighbors(q, K)
    np.testing.assert_array_equal(got, nb["slot"])
    assert fallbacks < n // 4
    assert first_tier > n // 2

