"""Oracle vs the numbers and closed forms the paper prints (tests/golden/paper_facts.json).

Each test names the passage it pins.  Monte Carlo tests use uniform queries on
the K=(8,...,8) torus, where the lift sum equals the quotient-metric sum.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle

FACTS = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_facts.json")))
K8 = (8,) * 8


@pytest.fixture(scope="module")
def mc():
    rng = np.random.default_rng(20210707)
    q = (rng.random((40000, 8)) * 8).astype(np.float32)
    return oracle.neighbors(q, K8)


def test_mean_support_matches_table1(mc):
    """Sec. 2.4, Table 1: average points in kernel support 64.94 (= 2 pi^4 / 3,
    ball volume over det Lambda)."""
    mean = mc["count"].mean()
    assert abs(mean - FACTS["table1_e8_average_points_in_support"]["value"]) < 0.25
    assert abs(2 * math.pi ** 4 / 3 - 64.94) < 0.005


def test_support_bounds_table1(mc):
    """Sec. 2.4, Table 1: max 121 (analytic), min 45 (Monte Carlo)."""
    assert mc["count"].max() <= FACTS["table1_e8_maximum_points_in_support"]["value"]
    assert mc["count"].min() >= FACTS["table1_e8_minimum_points_in_support_mc"]["value"]


def test_max_support_121_next_to_lattice_point():
    """Table 1's maximum: a query a hair away from a lattice point sees the point
    itself and exactly half of its 240 nearest neighbours (Sec. 2.5: they sit at
    distance sqrt 8).  The offset is 2^-9 times the E8 Weyl vector
    rho = (0,1,2,3,4,5,6,23) (or a signed permutation of it): |<rho, p>| >= 2 for
    every neighbour p at this scale, so each antipodal pair splits cleanly and
    the margin (~5e-3 in r^2) dwarfs fp32 rounding."""
    rng = np.random.default_rng(5)
    rho = np.array([0, 1, 2, 3, 4, 5, 6, 23], np.float64)
    bases = np.array([[2, 4, 0, 6, 2, 8, 4, 2], [1, 3, 5, 7, 1, 3, 5, 7], [0] * 8,
                      [14, 2, 2, 2, 2, 2, 2, 2]], np.float64)
    qs = []
    for b in bases:
        assert b.sum() % 4 == 0 and len(set(b % 2)) == 1
        for _ in range(3):
            v = rho[rng.permutation(8)] * np.where(rng.random(8) < 0.5, -1, 1)
            qs.append((b + 2.0 ** -9 * v) / 2)
    nb = oracle.neighbors(np.mod(np.array(qs), 8).astype(np.float32), K8)
    assert np.all(nb["count"] == FACTS["table1_e8_maximum_points_in_support"]["value"])


def test_total_weight_bounds(mc):
    """Sec. 2.5: (22158 - 625 sqrt 5)/24389 <= total weight <= 1; its mean over a
    uniform query is pi^4/105 (integral of f over R^8 divided by det Lambda = 256)."""
    f = FACTS["total_weight_lower_bound"]
    lo = (f["numerator_int"] + f["numerator_sqrt5_coeff"] * math.sqrt(5)) / f["denominator"]
    assert abs(lo - f["approx"]) < 5e-4
    w = mc["wsum"]
    assert w.min() >= lo - 1e-9
    assert w.max() <= FACTS["total_weight_upper_bound"]["value"] + 1e-12
    assert abs(w.mean() - math.pi ** 4 / 105) < 2e-3


def test_total_weight_one_at_lattice_points_and_deep_holes():
    """Sec. 2.5: total weight exactly 1 at lattice points and deep holes."""
    pts = np.array([
        [0, 0, 0, 0, 0, 0, 0, 0],
        [1, 1, 1, 1, 1, 1, 1, 1],          # odd coset point (sum 8)
        [2, 2, 0, 0, 0, 0, 0, 0],
        [2, 0, 0, 0, 0, 0, 0, 0],          # deep hole
        [1, 1, 1, 1, 1, 1, 1, -1],         # deep hole: (1^7,-1), sum 6
        [4, 2, 0, 0, 0, 0, 0, 0],          # deep hole translate
    ], np.float32) / 2
    nb = oracle.neighbors(np.mod(pts, 8), K8)
    assert np.all(nb["wsum"] == 1.0)
    assert list(nb["count"]) == [1, 1, 1, 16, 16, 16]


def test_lattice_point_returns_its_value():
    """Sec. 2.5: phi(k) = v_k -- one neighbour, weight exactly 1."""
    rng = np.random.default_rng(9)
    K = (4,) * 8
    N = 4 ** 8
    table = rng.standard_normal((N, 16))
    k = np.array([[0, 2, 2, 0, 0, 0, 0, 0], [1, 1, 1, 1, 1, 1, 1, 1], [3, -1, 1, 1, 1, 1, 1, 1]], np.int32)
    nb = oracle.neighbors((k / 2).astype(np.float32), K)
    out = oracle.forward(nb, oracle.gather_rows(table, nb["slot"]))
    np.testing.assert_array_equal(out, table[oracle.locations(k, K)])


def test_deep_hole_sixteen_sixteenths():
    """Sec. 2.5: at a deep hole (distance 2 = covering radius, Sec. 2.4) 16 points
    each get (1 - 4/8)^4 = 1/16."""
    nb = oracle.neighbors(np.array([[1, 0, 0, 0, 0, 0, 0, 0]], np.float32), K8)
    assert nb["count"][0] == 16
    assert np.all(nb["d2"][0, :16] == 4.0)
    assert np.all(nb["w64"][0, :16] == 1.0 / 16)
    assert np.all(nb["slot"][0, 16:] == -1)


def test_covering_radius(mc):
    """Sec. 2.4: covering radius 2 -- the closest point is never farther than 2."""
    assert mc["d2"][:, 0].max() <= FACTS["lambda_covering_radius"]["value"] ** 2
    # packing radius sqrt 2: two lattice points are >= sqrt 8 apart, so at most one
    # lies strictly inside distance sqrt 2
    assert np.all(mc["d2"][:, 1] >= 2.0)


def test_top32_weight_share(mc):
    """Sec. 2.6: the closest 32 points carry 99.5% of the weight on average, >= 90% always."""
    share = mc["w64"].sum(1) / mc["wsum"]
    assert abs(share.mean() - FACTS["top32_mean_weight_share"]["value"]) < 2e-3
    assert share.min() >= FACTS["top32_min_weight_share"]["value"]


def test_nearest_neighbour_shell_is_240():
    """E8 kissing number: 240 lattice points at distance sqrt 8 (Sec. 2.5).  A query
    at the midpoint of a lattice point and one neighbour has those two at d2 = 2;
    here we count the points at d2 = 8 from a lattice point via the oracle's
    recipe helper over the explicit shell."""
    shell = []
    for s in range(256):
        v = np.array([1 if (s >> i) & 1 else -1 for i in range(8)])
        if (v < 0).sum() % 2 == 0:
            shell.append(v)
    for i in range(8):
        for j in range(i + 1, 8):
            for a in (-2, 2):
                for b in (-2, 2):
                    v = np.zeros(8, int)
                    v[i], v[j] = a, b
                    shell.append(v)
    shell = np.array(shell, np.int32)
    assert shell.shape[0] == 240
    d = oracle.recipe_d2(np.zeros((240, 8), np.float32), shell)
    assert np.all(d == 8.0)
    # the query just off the origin (along the Weyl vector) sees exactly half of them
    rho = np.array([0, 1, 2, 3, 4, 5, 6, 23], np.float32)
    nb = oracle.neighbors((2.0 ** -10 * rho)[None, :], K8)
    assert nb["count"][0] == 121
    inside = nb["lift"][0, 1:121]
    assert np.all((inside[:, None, :] == shell[None, :, :]).all(-1).any(1))


def test_truncation_never_exceeds_32(mc):
    assert np.all((mc["slot"] >= 0).sum(1) == np.minimum(mc["count"], 32))


def test_recipe_weight_is_the_kernel():
    """Sec. 2.5: the fp32 weight the oracle records beside the fp64 one (the
    weight the GPU's selection and scatter use) is the kernel
    f(r) = (1 - r^2/8)^4 of that passage:
      * exactly 1 at a lattice point, and exactly 1/16 at each of the 16 points
        around a deep hole (the two special cases Sec. 2.5 names);
      * on queries of a 2^-3 grid at the doubled scale every squared distance
        is a multiple of 1/64, so u = 1 - r^2/8 = a/512 and u^2 are exact in
        fp32 and f(r) = a^4/2^36 is formed by one rounding: the recorded
        weight equals f(r) computed here from the lattice points in exact
        integers, rounded once to fp32;
      * elsewhere it stays within 4e-6 of f(r) taken in fp64 from the query and
        the listed lattice points (the fp32 differences, squares and sums of
        r^2 add at most 10 roundings of r^2 <= 8, i.e. 4.8e-6 in r^2, 6e-7 in
        u, and d(u^4)/du <= 4 over [0, 1], plus two roundings of the powers)."""
    pts = np.array([[0, 0, 0, 0, 0, 0, 0, 0], [1, 1, 1, 1, 1, 1, 1, 1], [2, 0, 0, 0, 0, 0, 0, 0],
                    [1, 1, 1, 1, 1, 1, 1, -1]], np.float32) / 2
    nb = oracle.neighbors(np.mod(pts, 8), K8)
    assert nb["w32"][0, 0] == 1.0 and nb["w32"][1, 0] == 1.0
    assert np.all(nb["w32"][:2, 1:] == 0.0)
    assert np.all(nb["w32"][2:, :16] == np.float32(1.0 / 16)) and np.all(nb["w32"][2:, 16:] == 0.0)

    rng = np.random.default_rng(2107)
    grid = rng.integers(0, 8 * 16, size=(400, 8))            # x = grid / 8 on [0, 16)
    nb = oracle.neighbors((grid / 16.0).astype(np.float32), K8)
    valid = nb["slot"] >= 0
    e8 = grid[:, None, :] - 8 * nb["lift"].astype(np.int64)   # 8 (x - k), exact integers
    r2_64 = (e8 * e8).sum(-1)                                  # 64 r^2
    a = 512 - r2_64                                            # 512 u
    assert np.all(a[valid] > 0)
    exact = (a.astype(np.float64) ** 4 / 2.0 ** 36).astype(np.float32)
    np.testing.assert_array_equal(nb["w32"][valid], exact[valid])
    assert np.unique(a[valid]).size > 100                      # many distinct weights covered

    q = (rng.random((2000, 8)) * 8).astype(np.float32)
    nb = oracle.neighbors(q, K8)
    valid = nb["slot"] >= 0
    e = nb["x"].astype(np.float64)[:, None, :] - nb["lift"].astype(np.float64)
    f = (1.0 - (e * e).sum(-1) / 8.0) ** 4
    assert np.abs(nb["w32"][valid] - f[valid]).max() <= 4e-6
