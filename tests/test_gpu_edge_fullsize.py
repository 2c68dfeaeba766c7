"""The method's special queries in the benchmark's launch configuration.

One batch of 262,144 lookups on K = (8, ..., 8), m = 32 -- 64 lookups per wave,
the forward's two-deep pipeline and the merged scatter's 64-lookup batches --
with the exceptional queries of Sec. 2.5 / 2.6 placed at every wave position
t in [0, 64): lattice points (one neighbour), deep holes (16 at weight 1/16),
points a hair from a lattice point (the shell at r^2 = 8 - O(10^-7), where
rounding decides), dyadic queries (exact distance ties at the 32nd place),
out-of-range and negative copies of them, and non-finite queries.  A uniform
variant and a clustered one (the specials sit in the clusters' cells, so the
merged scatter merges batches that hold them).  Every output, every dq and
every touched value-gradient row is compared with the oracle in the atomic,
sorted and merged modes (dV against the fp64 sums of the recipe weights, the
weights the lists pin bit-exactly: next to a lattice point the shell points'
weights are ~1e-28 and can be a row's only contribution); rows no lookup
touches stay exactly 0.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
import paper_2107_03474_amd as lram
from test_gpu_parity import _rel_rows, special_queries

pytestmark = pytest.mark.gpu
DEV = "cuda"
K8 = (8,) * 8
L = 262144


def _say(*a):
    print(*a, flush=True)


def _specials(rng, centres):
    """About 60 exceptional queries (user scale), some next to the given centres."""
    sp = [special_queries(K8)]
    rho = np.array([0, 1, 2, 3, 4, 5, 6, 23], np.float64)
    for c in centres:
        k = 2 * np.round(c)                                 # a point of 2 Z^8 ...
        if k.sum() % 4:                                     # ... with coordinate sum 0 mod 4
            k[0] += 2
        pts = [k, k + np.r_[2.0, np.zeros(7)],              # lattice point, deep hole
               k + 1e-6 * rng.standard_normal(8),           # shell at the support edge
               k + 2.0 ** -9 * rho[rng.permutation(8)],     # 121 points in the support
               np.round(2 * c * 4) / 4]                     # dyadic: ties
        sp.append(np.mod(np.array(pts) / 2, 8))
    sp.append(np.array([[np.nan] * 8, [0, np.inf, 0, 0, 0, 0, 0, 0], [0, 0, -np.inf, 0, 0, 0, 0, 0],
                        [3e38, 0, 0, 0, 0, 0, 0, 1]]))
    return np.concatenate(sp).astype(np.float32)


def _batch(clustered):
    rng = np.random.default_rng(77 if clustered else 78)
    centres = rng.random((5, 8)) * 8
    q = rng.random((L, 8)) * 8
    if clustered:
        hot = rng.random(L) < 0.8
        q[hot] = np.mod(centres[rng.integers(0, 5, hot.sum())] + 0.3 * rng.standard_normal((hot.sum(), 8)), 8)
    q = q.astype(np.float32)
    q = np.where(q >= 8, np.float32(0), q)
    sp = _specials(rng, centres)
    assert sp.shape[0] <= 64
    for i in range(sp.shape[0]):
        for t in range(64):
            q[64 * (64 * i + t) + t] = sp[i]                # wave 64 i + t, position t
    return q


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("clustered", [False, True])
def test_special_queries_at_every_wave_position(clustered, dtype):
    _say("edge cases at full launch size: clustered=%s %s" % (clustered, dtype))
    q_np = _batch(clustered)
    q = torch.from_numpy(q_np).to(DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(79)
    table = (torch.randn((8 ** 8, 32), generator=g, device=DEV) * 0.02).to(dtype)
    G = torch.randn((L, 32), generator=g, device=DEV)
    out = lram.forward(q, table, K8)
    slot, _, _ = lram.neighbors(q, K8, want_d2=False)
    torch.cuda.synchronize()
    nb = oracle.neighbors(q_np, K8)
    assert np.array_equal(slot.cpu().numpy(), nb["slot"])
    assert (nb["count"] < 32).sum() >= 64 * 10              # the specials are in the batch
    rows = oracle.gather_rows(table.float().cpu().numpy(), nb["slot"])
    err = _rel_rows(out.float().cpu().numpy(), oracle.forward(nb, rows))
    _say("out: max rel err %.2e" % err.max())
    assert err.max() <= (1e-5 if dtype == torch.float32 else 2e-2)
    Gn = G.cpu().numpy()
    dq_ref = oracle.grad_query(nb, rows, Gn)
    del rows
    uniq, acc = oracle.grad_table_rows(nb, Gn, weights="w32")
    ut = torch.from_numpy(uniq).to(DEV)
    touched = torch.zeros(8 ** 8, dtype=torch.bool, device=DEV)
    touched[ut] = True
    dq0 = None
    for mode in ("atomic", "sorted", "merged"):
        gt, gq = lram.backward(q, table, K8, G, mode=mode)
        torch.cuda.synchronize()
        if dq0 is None:
            err = _rel_rows(gq.cpu().numpy(), dq_ref)
            _say("dq: max rel err %.2e" % err.max())
            assert err.max() <= 1e-5
            dq0 = gq
        else:
            assert torch.equal(gq, dq0), mode            # dq does not depend on the scatter
        err = _rel_rows(gt[ut].cpu().numpy(), acc)
        _say("dV (%s): max rel err %.2e over %d rows" % (mode, err.max(), uniq.size))
        assert err.max() <= 1e-5
        assert torch.count_nonzero(gt[~touched]).item() == 0
        del gt, gq
        gc.collect()
        torch.cuda.empty_cache()
    if clustered:
        assert lram.resolved_mode(L, 1, "auto") == "merged"
