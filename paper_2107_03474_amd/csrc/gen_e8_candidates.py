#!/usr/bin/env python3
"""Generate the E8 candidate table used by the GPU neighbour search.

Sec. 2.6 of the paper maps a query by a lattice isometry into the fundamental
region

    F = { z : z_0 >= z_1 >= ... >= z_6 >= |z_7|,  z_0 + z_1 <= 2,  sum z <= 4 }

(Lambda = 2*E8 scale) and scans a fixed list of lattice points: those whose
distance to F is below sqrt(8).  This script finds that list by convex
quadratic programming, done exactly: the projection of a point p onto F is the
projection onto the affine span of some active set S of F's ten facets with
non-negative multipliers; all 2^10 active sets are tried (vectorised fp64),
and every classification near r^2 = 8 is re-derived in exact rational
arithmetic.

Output (``e8_candidates.inc``):
  * the STRICT list  -- dist(p, F)^2 < 8 (the paper's 232 points), in
    ascending order of that distance, and E8_FAST / E8_FAST_BOUND: the first
    E8_FAST of them and the exact distance^2 from F of every later one, at
    least E8_FAST_BOUND (a query in F whose k-th closest point among the
    first E8_FAST lies below that bound takes its closest k from them), and
    the same for the first E8_FAST2 (E8_FAST2_BOUND), a smaller first tier;
  * the BOUNDARY list -- dist(p, F)^2 == 8 exactly.  These never lie in the open
    support of a query inside F, but a query whose reduction lands a rounding
    error outside F, or whose fp32 distance rounds below 8, can see them; the
    kernel scans them only on that rare path.
The gap to the next distance level is checked to be large.
"""
from __future__ import annotations

import os
import sys
from fractions import Fraction

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "e8_candidates.inc")


FAST = 192  # three candidates per lane of a 64-lane wave
FAST2 = 128  # two per lane: the first tier of the fast set


def lattice_points(max_norm: int) -> np.ndarray:
    """All points of Lambda = {x in (2Z)^8 u (2Z+1)^8 : sum x = 0 mod 4} with |x|^2 <= max_norm."""
    r = int(np.floor(np.sqrt(max_norm)))
    pts = []
    for eps in (0, 1):
        vals = np.array([v for v in range(-r, r + 1) if (v - eps) % 2 == 0], np.int64)
        grid = np.stack(np.meshgrid(*([vals] * 8), indexing="ij"), -1).reshape(-1, 8)
        keep = ((grid * grid).sum(1) <= max_norm) & (grid.sum(1) % 4 == 0)
        pts.append(grid[keep])
    return np.concatenate(pts)


def facets():
    """F as A z <= b (10 rows)."""
    A, b = [], []
    for j in range(6):
        row = np.zeros(8, np.int64)
        row[j + 1], row[j] = 1, -1
        A.append(row), b.append(0)
    row = np.zeros(8, np.int64); row[7], row[6] = 1, -1; A.append(row); b.append(0)
    row = np.zeros(8, np.int64); row[7], row[6] = -1, -1; A.append(row); b.append(0)
    row = np.zeros(8, np.int64); row[0] = row[1] = 1; A.append(row); b.append(2)
    A.append(np.ones(8, np.int64)); b.append(4)
    return np.array(A), np.array(b)


def project_all(P: np.ndarray):
    """fp64 distance^2 from every row of P to F and the active set achieving it."""
    A, b = facets()
    best = np.full(P.shape[0], np.inf)
    best_set = [None] * P.shape[0]
    Pf = P.astype(np.float64)
    for mask in range(1 << 10):
        S = [i for i in range(10) if mask >> i & 1]
        if S:
            As = A[S].astype(np.float64)
            G = As @ As.T
            if np.linalg.matrix_rank(G) < len(S):
                continue
            lam = np.linalg.solve(G, (As @ Pf.T) - b[S][:, None].astype(np.float64))  # [|S|, n]
            Z = Pf - (As.T @ lam).T
            ok = np.all(lam >= -1e-9, axis=0)
        else:
            Z = Pf.copy()
            ok = np.ones(P.shape[0], bool)
        feas = np.all(A @ Z.T <= b[:, None] + 1e-9, axis=0)
        ok &= feas
        d = ((Pf - Z) ** 2).sum(1)
        upd = ok & (d < best - 1e-12)
        best[upd] = d[upd]
        for i in np.nonzero(upd)[0]:
            best_set[i] = S
    return best, best_set


def exact_dist2(p, S) -> Fraction:
    """Exact KKT check of active set S for point p; returns dist^2 as a Fraction."""
    A, b = facets()
    p = [Fraction(int(v)) for v in p]
    if not S:
        z = p
        lam = []
    else:
        As = [[Fraction(int(v)) for v in A[i]] for i in S]
        n = len(S)
        G = [[sum(As[i][k] * As[j][k] for k in range(8)) for j in range(n)] for i in range(n)]
        rhs = [sum(As[i][k] * p[k] for k in range(8)) - b[S[i]] for i in range(n)]
        # Gaussian elimination in rationals
        M = [G[i][:] + [rhs[i]] for i in range(n)]
        for c in range(n):
            piv = next(r for r in range(c, n) if M[r][c] != 0)
            M[c], M[piv] = M[piv], M[c]
            for r in range(n):
                if r != c and M[r][c] != 0:
                    f = M[r][c] / M[c][c]
                    M[r] = [M[r][k] - f * M[c][k] for k in range(n + 1)]
        lam = [M[i][n] / M[i][i] for i in range(n)]
        z = [p[k] - sum(lam[i] * As[i][k] for i in range(n)) for k in range(8)]
    assert all(l >= 0 for l in lam), "negative multiplier"
    for i in range(10):
        assert sum(Fraction(int(A[i][k])) * z[k] for k in range(8)) <= b[i], "infeasible"
    return sum((p[k] - z[k]) ** 2 for k in range(8))


def main(write: bool = True) -> dict:
    # |z| <= 2 on F (covering radius), so a point within sqrt 8 of F has |p|^2 < (2 + sqrt 8)^2 < 24;
    # norm 24 is included to measure the gap above the boundary level.
    P = lattice_points(24)
    d2, sets = project_all(P)
    strict, boundary, above = [], [], []
    for i in range(P.shape[0]):
        if d2[i] > 8 + 1e-6 and d2[i] > 9.0:
            above.append(d2[i])
            continue
        ex = exact_dist2(P[i], sets[i])
        if ex < 8:
            strict.append((ex, P[i]))
        elif ex == 8:
            boundary.append(P[i])
        else:
            above.append(float(ex))
    strict = sorted(strict, key=lambda e: (e[0], int((e[1] * e[1]).sum()), tuple(-e[1])))
    strict_d2 = [e[0] for e in strict]
    strict = [e[1] for e in strict]
    fast_bound = strict_d2[FAST] if FAST < len(strict) else Fraction(8)
    fast2_bound = strict_d2[FAST2]
    boundary = sorted(boundary, key=lambda v: (int((v * v).sum()), tuple(-v)))
    gap = min(above) - 8.0
    norms = {}
    for v in strict:
        norms[int((v * v).sum())] = norms.get(int((v * v).sum()), 0) + 1
    allpts = np.array(strict + boundary)
    info = dict(strict=np.array(strict), boundary=np.array(boundary), gap=gap, norms=norms,
                cmin=int(allpts.min()), cmax=int(allpts.max()), strict_d2=strict_d2, fast_bound=fast_bound,
                fast2_bound=fast2_bound)
    if write:
        with open(OUT, "w") as f:
            f.write("// Generated by gen_e8_candidates.py -- do not edit.\n")
            f.write("// Lattice points of Lambda = 2*E8 by their exact distance to the fundamental\n")
            f.write("// region F (Sec. 2.6): STRICT: dist^2 < 8, BOUNDARY: dist^2 == 8.\n")
            f.write("// Next distance^2 level above 8: 8 + %.6f.\n" % gap)
            f.write("#pragma once\n")
            f.write("#define E8_NSTRICT %d\n#define E8_NBOUNDARY %d\n" % (len(strict), len(boundary)))
            f.write("#define E8_CAND_MIN %d\n#define E8_CAND_MAX %d\n" % (info["cmin"], info["cmax"]))
            f.write("// Strict points FAST.. lie at distance^2 >= %s from F.\n" % fast_bound)
            f.write("#define E8_FAST %d\n#define E8_FAST_BOUND %.9gf\n" % (FAST, float(fast_bound)))
            f.write("// Strict points FAST2.. lie at distance^2 >= %s from F.\n" % fast2_bound)
            f.write("#define E8_FAST2 %d\n#define E8_FAST2_BOUND %.9gf\n" % (FAST2, float(fast2_bound)))
            for name, lst in (("E8_STRICT_INIT", strict), ("E8_BOUNDARY_INIT", boundary)):
                f.write("#define %s { \\\n" % name)
                for v in lst:
                    f.write("  {%s}, \\\n" % ", ".join("%2d" % int(c) for c in v))
                f.write("}\n")
    return info


if __name__ == "__main__":
    info = main(write="--check" not in sys.argv)
    print("strict", len(info["strict"]), "by norm", info["norms"], "boundary", len(info["boundary"]),
          "gap", info["gap"], "coord range", info["cmin"], info["cmax"])
