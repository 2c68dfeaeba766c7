"""All-locations brute force for tiny tori -- a pin for the oracle.

It shares nothing with the oracle's enumeration: instead of walking lattice
points coordinate by coordinate, it lists every memory location of the torus
(every coset representative k = 2Y + eps of Lambda / L_K, Sec. 2.2 and Sec. 2.4),
then every lift k + 2K*n of each location that lies within sqrt(8) of the
query in each coordinate, and keeps the lifts whose fp32 recipe distance is
below 8 (Sec. 2.5).  The location index is computed from (eps, Y) directly.
Affordable for N up to ~1e5 locations.
"""
from __future__ import annotations

import itertools

import numpy as np

R = 2.8284271247461903


def all_locations(K):
    """(k [N,8] int64 representatives in [0,2K), slot [N] int64) for every location."""
    K = np.asarray(K, np.int64)
    N = int(np.prod(K))
    Y = np.stack(np.meshgrid(*[np.arange(k) for k in K], indexing="ij"), -1).reshape(-1, 8)
    Y = Y[Y.sum(1) % 2 == 0]
    reps, slots = [], []
    for eps in (0, 1):
        k = 2 * Y + eps
        idx = Y[:, 0].copy()
        for i in range(1, 7):
            idx = idx * K[i] + Y[:, i]
        idx = idx * (K[7] // 2) + Y[:, 7] // 2
        reps.append(k)
        slots.append(eps * (N // 2) + idx)
    k = np.concatenate(reps)
    s = np.concatenate(slots)
    assert k.shape[0] == N
    return k, s


def recipe_d2(x: np.ndarray, k: np.ndarray) -> np.ndarray:
    """fp32 distance recipe, vectorised over rows of k (x is one query)."""
    e = x[None, :].astype(np.float32) - k.astype(np.float32)
    sq = e * e
    s = sq[:, 0].copy()
    for i in range(1, 8):
        s = s + sq[:, i]
    return s


def support(x: np.ndarray, K, locs=None):
    """All lifts with recipe distance < 8 around the Lambda-scale query x (fp32).

    Returns (d2 [n] fp32, slot [n], lift [n,8]) sorted by (bits(d2), slot, lift)."""
    K = np.asarray(K, np.int64)
    if locs is None:
        locs = all_locations(K)
    reps, slots = locs
    x = np.asarray(x, np.float32)
    xd = x.astype(np.float64)
    # per coordinate: the lifts of each representative value within sqrt(8)
    per_coord = []
    for i in range(8):
        shifts = np.arange(-3, 4) * 2 * K[i]
        cand = reps[:, i][:, None] + shifts[None, :]
        ok = np.abs(xd[i] - cand) < R + 1e-3
        per_coord.append((cand, ok))
    maxc = max(int(ok.sum(1).max()) for _, ok in per_coord)
    # list lift options per coordinate as (value, present) padded to maxc
    opts = []
    for cand, ok in per_coord:
        order = np.argsort(~ok, axis=1, kind="stable")
        vals = np.take_along_axis(cand, order, 1)[:, :maxc]
        pres = np.take_along_axis(ok, order, 1)[:, :maxc]
        opts.append((vals, pres))
    d_all, s_all, k_all = [], [], []
    for combo in itertools.product(range(maxc), repeat=8):
        present = np.ones(reps.shape[0], bool)
        k = np.empty_like(reps)
        for i, c in enumerate(combo):
            present &= opts[i][1][:, c]
            k[:, i] = opts[i][0][:, c]
        if not present.any():
            continue
        kk = k[present]
        d = recipe_d2(x, kk)
        keep = d < np.float32(8.0)
        d_all.append(d[keep])
        s_all.append(slots[present][keep])
        k_all.append(kk[keep])
    d = np.concatenate(d_all) if d_all else np.zeros(0, np.float32)
    s = np.concatenate(s_all) if s_all else np.zeros(0, np.int64)
    k = np.concatenate(k_all) if k_all else np.zeros((0, 8), np.int64)
    bits = d.view(np.uint32).astype(np.int64)
    order = np.lexsort(tuple(k[:, i] for i in range(7, -1, -1)) + (s, bits))
    return d[order], s[order], k[order]
