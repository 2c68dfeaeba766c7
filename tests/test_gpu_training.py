"""GPU parity of the access statistics and the sparse Adam step against the oracle.

Bars: the weighted access histogram per location relative <= 1e-5 (fp32
atomics against the fp64 sum of the recipe weights), the set of accessed
locations exact, the KL divergence relative <= 1e-6; a lattice-point batch
gives used = 1 and KL = 0.  Adam: moments per row relative <= 1e-6, the step
(new - old value) per row relative <= 1e-4 (fp32 table entries of size 0.02
carry 2e-9 of rounding against steps of size lr), bf16 tables within one bf16
unit of the rounded fp64 result plus the fp32 rounding of the step; untouched
rows bit-identical; used gradient rows cleared.  The touched-row step
(flags from lram_mark_touched) is bit-identical to the full-scan step on
table, moments and gradient, and leaves every flag cleared; the flags mark
exactly the oracle's locations of the lookups.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
import paper_2107_03474_amd as lram
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _rel_rows(a, b):
    a = np.asarray(a, np.float64).reshape(a.shape[0], -1)
    b = np.asarray(b, np.float64).reshape(b.shape[0], -1)
    num = np.linalg.norm(a - b, axis=1)
    den = np.linalg.norm(b, axis=1)
    return np.where(den > 0, num / np.where(den > 0, den, 1), num)


@pytest.mark.parametrize("K", [(4, 4, 4, 4, 8, 8, 8, 8), (2, 4, 6, 8, 2, 4, 6, 8)])
def test_access_stats(K):
    N = int(np.prod(K))
    w = W.Workload("t", K, 32, "f32", 4096, 4, "zipf_mix", False, gmm_sigma=0.3, zipf_centres=64, zipf_s=1.1)
    q_np = W.queries(w).reshape(-1, 8)
    q = torch.from_numpy(q_np).to(DEV)
    hist = lram.access_histogram(q, K)
    st = lram.access_stats(hist)
    nb = oracle.neighbors(q_np, K)
    href = oracle.access_histogram(nb, N, weights="w32")
    h = hist.cpu().numpy().astype(np.float64)
    assert np.array_equal(h > 0, href > 0)
    np.testing.assert_allclose(h[href > 0], href[href > 0], rtol=1e-5)
    used, kl = oracle.access_stats(oracle.access_histogram(nb, N))
    assert st["count"] == int((href > 0).sum()) and abs(st["used"] - used) < 1e-15
    np.testing.assert_allclose(st["kl"], kl, rtol=1e-6)


def test_access_stats_lattice_points_uniform():
    K = (2, 2, 2, 4, 2, 2, 2, 2)
    pts = []
    for eps in (0, 1):
        for Y in itertools.product(*[range(k) for k in K]):
            if sum(Y) % 2 == 0:
                pts.append((2 * np.asarray(Y) + eps) / 2.0)
    q = torch.from_numpy(np.asarray(pts, np.float32)).to(DEV)
    st = lram.access_stats(lram.access_histogram(q, K))
    assert st["used"] == 1.0 and abs(st["kl"]) < 1e-9 and st["count"] == int(np.prod(K))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("m", [32, 64])
def test_sparse_adam(m, dtype):
    rng = np.random.default_rng(5)
    N = 70001
    V0 = (rng.standard_normal((N, m)) * 0.02).astype(np.float32)
    g = rng.standard_normal((N, m)).astype(np.float32) * 1e-2
    g[rng.random(N) < 0.4] = 0.0          # untouched rows
    g[7, :5] = 0.0                         # a touched row with some zero entries
    m1 = (rng.standard_normal((N, m)) * 1e-3).astype(np.float32)
    m2 = (rng.random((N, m)) * 1e-4).astype(np.float32)
    table = torch.from_numpy(V0).to(DEV).to(dtype)
    V0r = table.float().cpu().numpy()       # the table as stored (bf16-rounded)
    grad = torch.from_numpy(g).to(DEV)
    e1 = torch.from_numpy(m1).to(DEV)
    e2 = torch.from_numpy(m2).to(DEV)
    lram.sparse_adam(table, grad, e1, e2, step=3, lr=1e-3)
    torch.cuda.synchronize()
    Vr, r1, r2 = oracle.sparse_adam(V0r, g, m1, m2, 3, lr=1e-3)
    touched = np.any(g != 0, axis=1)
    Vg = table.float().cpu().numpy()
    assert np.array_equal(Vg[~touched], V0r[~touched])
    assert np.array_equal(e1.cpu().numpy()[~touched], m1[~touched])
    assert np.array_equal(e2.cpu().numpy()[~touched], m2[~touched])
    assert _rel_rows(e1.cpu().numpy()[touched], r1[touched]).max() <= 1e-6
    assert _rel_rows(e2.cpu().numpy()[touched], r2[touched]).max() <= 1e-6
    if dtype == torch.float32:
        assert _rel_rows((Vg - V0r)[touched], (Vr - V0r)[touched]).max() <= 1e-4
    else:
        ref = torch.from_numpy(Vr.astype(np.float32)).to(torch.bfloat16).float().numpy()
        # one bf16 unit at either magnitude, plus the fp32 rounding of the step
        # (which dominates where the step cancels the value)
        bound = np.maximum(np.abs(ref), np.abs(Vg)) * 2.0 ** -7 + 4 * 2.0 ** -24 * np.abs(Vr - V0r) + 1e-30
        assert np.all(np.abs(Vg[touched] - ref[touched]) <= bound[touched])
    assert torch.count_nonzero(grad).item() == 0


def test_training_step_roundtrip():
    """forward + backward (merged) + the Adam step leave untouched rows alone
    and move exactly the rows the batch read."""
    K = (4, 4, 4, 4, 8, 8, 8, 8)
    N = int(np.prod(K))
    rng = np.random.default_rng(6)
    q = torch.from_numpy((rng.random((140000, 8)) * np.asarray(K)).astype(np.float32)).to(DEV)
    table = (torch.randn((N, 64), device=DEV) * 0.02)
    before = table.clone()
    opt = lram.SparseAdam(table, lr=1e-3)
    G = torch.randn((140000, 64), device=DEV)
    gt, _ = lram.backward(q, table, K, G, want_grad_q=False, mode="merged")
    read = torch.zeros(N, dtype=torch.bool, device=DEV)
    s = lram.neighbors(q, K, want_d2=False)[0]
    read[s[s >= 0].long()] = True
    opt.step(gt)
    torch.cuda.synchronize()
    moved = (table != before).any(1)
    assert torch.equal(moved, read)
    assert torch.count_nonzero(gt).item() == 0


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("m", [32, 64])
def test_sparse_adam_touched_matches_full_scan(m, dtype):
    K = (4, 4, 4, 4, 8, 8, 8, 8)
    N = int(np.prod(K))
    rng = np.random.default_rng(8)
    q_np = (rng.random((3000, 8)) * np.asarray(K)).astype(np.float32)
    q_np[7] = np.nan                       # no neighbours
    q = torch.from_numpy(q_np).to(DEV)
    touched = lram.mark_touched(q, K)
    nb = oracle.neighbors(q_np, K)
    ref = np.zeros(N, bool)
    ref[nb["slot"][nb["slot"] >= 0]] = True
    assert np.array_equal(touched.cpu().numpy() != 0, ref)
    table = (torch.randn((N, m), device=DEV) * 0.02).to(dtype)
    G = torch.randn((3000, m), device=DEV)
    G[11] = 0.0                            # a lookup whose rows get no gradient from it
    gt, _ = lram.backward(q, table.float() if dtype == torch.float32 else table, K, G, want_grad_q=False,
                          mode="merged")
    e1 = (torch.randn((N, m), device=DEV) * 1e-3)
    e2 = torch.rand((N, m), device=DEV) * 1e-4
    t2, g2, a1, a2 = table.clone(), gt.clone(), e1.clone(), e2.clone()
    lram.sparse_adam(table, gt, e1, e2, step=5, lr=1e-3)
    lram.sparse_adam(t2, g2, a1, a2, step=5, lr=1e-3, touched=touched)
    torch.cuda.synchronize()
    assert torch.equal(table, t2) and torch.equal(e1, a1) and torch.equal(e2, a2) and torch.equal(gt, g2)
    assert torch.count_nonzero(touched).item() == 0
