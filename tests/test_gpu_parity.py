"""GPU parity: the HIP library (through the C ABI) against the oracle.

Bars (fixed before any kernel ran):
  * neighbour locations: bit-exact, in selection order; recipe distances and
    recipe weights: bit-exact (they are decided in the same fp32 arithmetic);
  * forward, per output row: relative L2 error <= 1e-5 for fp32 tables and
    <= 2e-2 for bf16 tables (the output is rounded to bf16 once), against the
    fp64 oracle;
  * dq and the value-gradient rows (fp32 outputs for either table dtype, whose
    bf16 entries are exact in fp32): relative L2 error <= 1e-5;
  * value-gradient rows no lookup touched stay exactly 0.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2107_03474_amd as lram
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _say(*a):
    print(*a, flush=True)


def _rel_rows(a, b):
    """Per-row relative L2 error of a against reference b (rows with |b| = 0 use |a|)."""
    a = np.asarray(a, np.float64).reshape(a.shape[0], -1)
    b = np.asarray(b, np.float64).reshape(b.shape[0], -1)
    num = np.linalg.norm(a - b, axis=1)
    den = np.linalg.norm(b, axis=1)
    return np.where(den > 0, num / np.where(den > 0, den, 1), num)


def check_neighbors(q_np, K):
    q = torch.from_numpy(np.ascontiguousarray(q_np)).to(DEV)
    slot, w, d2 = lram.neighbors(q, K)
    torch.cuda.synchronize()
    nb = oracle.neighbors(q_np, K)
    s = slot.cpu().numpy().reshape(nb["slot"].shape)
    bad = np.nonzero((s != nb["slot"]).any(-1).reshape(-1))[0]
    assert bad.size == 0, "first mismatching lookup %d: gpu %s oracle %s" % (
        bad[0], s.reshape(-1, 32)[bad[0]], nb["slot"].reshape(-1, 32)[bad[0]])
    np.testing.assert_array_equal(d2.cpu().numpy().reshape(nb["d2"].shape).view(np.uint32), nb["d2"].view(np.uint32))
    np.testing.assert_array_equal(w.cpu().numpy().reshape(nb["w32"].shape).view(np.uint32), nb["w32"].view(np.uint32))
    return nb


def special_queries(K):
    Kf = np.asarray(K, np.float64)
    rho = np.array([0, 1, 2, 3, 4, 5, 6, 23], np.float64)
    pts = [np.zeros(8), np.full(8, 0.5), [1, 0, 0, 0, 0, 0, 0, 0], [0.5] * 7 + [-0.5], 2.0 ** -11 * rho,
           np.full(8, 0.5) + 2.0 ** -11 * rho, [1, 1, 0, 0, 0, 0, 0, 0.0], [0.25, 0.25, 0.25, 0.25, 0, 0, 0, 0],
           [0.5, 0.5, 0.5, 0.5, 0.5, 0.5, 0.5, 1.0], [3, 1, 2, 0.5, 0.25, 0.125, 1.5, 2.5],
           -np.array([1.25, 0.5, 3.0, 0.75, 2.0, 1.0, 0.5, 0.25])]
    q = np.array(pts, np.float64)
    q = np.concatenate([q, q + Kf * 3, q - Kf])          # the same points seen through the wrap
    return q.astype(np.float32)


@pytest.mark.parametrize("K", [(4,) * 8, (8,) * 8, (12,) * 8, (14,) * 8, (2, 4, 6, 8, 10, 2, 4, 6), (2,) * 8])
def test_neighbors_random(K):
    _say("neighbors random K=%s" % (K,))
    rng = np.random.default_rng(7)
    q = (rng.random((2000, 8)) * np.asarray(K)).astype(np.float32)
    q[:200] = q[:200] * 5 - 2 * np.asarray(K, np.float32)   # out of range, negative
    check_neighbors(q, K)


@pytest.mark.parametrize("K", [(8192, 2, 4, 2, 2, 2, 2, 2), (2, 2, 2, 2, 2, 2, 2, 8192), (16,) * 7 + (6,)])
def test_neighbors_size_limits(K):
    """The largest torus side the library takes (K_i = 8192: Lambda-scale
    coordinates up to 2K = 16384, wrapped near both ends) and a torus with
    N = 1.61e9 locations, close to 2^31 (the location sums of the table build
    run in uint32 up to 2N)."""
    _say("neighbors size limits K=%s" % (K,))
    rng = np.random.default_rng(17)
    Kf = np.asarray(K, np.float64)
    q = rng.random((3000, 8)) * Kf
    q[:500] = np.where(rng.random((500, 8)) < 0.5, rng.random((500, 8)) * 2.0,
                       Kf - rng.random((500, 8)) * 2.0)     # next to the wrap on both sides
    q[500:600] = Kf - 1e-3 * rng.random((100, 8))
    q = q.astype(np.float32)
    q = np.where(q >= Kf.astype(np.float32), np.float32(0), q).astype(np.float32)
    nb = check_neighbors(q, K)
    assert nb["slot"].max() > int(np.prod(K)) * 0.99 or max(K) == 8192


@pytest.mark.parametrize("K", [(4,) * 8, (8,) * 8, (2, 2, 2, 2, 4, 4, 4, 4)])
def test_neighbors_special_points(K):
    _say("neighbors special K=%s" % (K,))
    nb = check_neighbors(special_queries(K), K)
    assert (nb["count"] < 32).any()


def test_neighbors_dyadic_grid():
    """Coarse dyadic queries produce many exact distance ties at the 32nd place."""
    _say("neighbors dyadic")
    rng = np.random.default_rng(8)
    K = (8,) * 8
    q = (rng.integers(0, 8 * 8, size=(3000, 8)) / 8.0).astype(np.float32)
    check_neighbors(q, K)


def _tier_band_queries(K, seed):
    """Queries for each path of the search's fast candidate set, chosen by the
    oracle's fp32 distance of the 32nd neighbour d: below the first tier's
    limit 48/7 - 2^-7 (band a), within 1e-3 of it, between it and the second
    tier's limit 15/2 - 2^-7 (band b), within 2e-3 of that, and above it or
    with fewer than 32 points in the support (the full scan).  Noise of
    0.05-0.1 around the deep holes spreads d over all of them."""
    rng = np.random.default_rng(seed)
    Kf = np.asarray(K, np.float64)
    holes = np.array([[1, 0, 0, 0, 0, 0, 0, 0.0], [0.5] * 8, [0.5] * 7 + [-0.5]])
    parts = [np.mod(h + 1.0 + sc * rng.standard_normal((1500, 8)), Kf) for h in holes for sc in (0.05, 0.1)]
    parts.append(rng.random((3000, 8)) * Kf)
    q = np.concatenate(parts).astype(np.float32)
    nb = oracle.neighbors(q, K)
    d = np.where(nb["count"] >= 32, nb["d2"][:, 31], np.inf)
    lim2 = np.float32(np.float32(48 / 7) - np.float32(2.0 ** -7))
    lim1 = np.float32(7.5 - 2.0 ** -7)
    bands = {"a": d < lim2 - 1e-3, "a|b": np.abs(d - lim2) < 1e-3, "b": (d >= lim2 + 1e-3) & (d < lim1 - 2e-3),
             "b|full": np.abs(d - lim1) < 2e-3, "full": d >= lim1 + 2e-3}
    pick = []
    for name, m in bands.items():
        idx = np.nonzero(m)[0]
        assert idx.size >= (5 if "|" in name else 100), (name, idx.size)
        pick.append(idx[:300])
    return q[np.concatenate(pick)]


@pytest.mark.parametrize("K", [(4,) * 8, (14,) * 8])
def test_neighbors_each_fast_tier(K):
    """Lists of queries taken by each tier of the fast candidate set, by the
    full scan, and at the tiers' edges: bit-exact locations, distances and
    weights; for the 4^8 torus also the forward in its full launch
    configuration (64 lookups per wave, lists double-buffered), with the
    queries spread over 262,144 lookups."""
    _say("neighbors per fast tier K=%s" % (K,))
    q_np = _tier_band_queries(K, 17)
    nb = check_neighbors(q_np, K)
    if K != (4,) * 8:
        return
    reps = -(-262144 // q_np.shape[0])
    perm = np.random.default_rng(4).permutation(reps * q_np.shape[0])
    idx = np.tile(np.arange(q_np.shape[0]), reps)[perm]
    table = _small_table(K, 32, torch.float32)
    out = lram.forward(torch.from_numpy(q_np[idx]).to(DEV), table, K)
    torch.cuda.synchronize()
    ref = oracle.forward(nb, oracle.gather_rows(table.cpu().numpy(), nb["slot"]))
    err = _rel_rows(out.cpu().numpy(), ref[idx])
    assert err.max() <= 1e-5, err.max()


def test_neighbors_nonfinite_and_ragged():
    _say("neighbors nonfinite/ragged")
    K = (4,) * 8
    rng = np.random.default_rng(9)
    for L in (1, 2, 63, 64, 65, 255, 257, 1000):
        q = (rng.random((L, 8)) * 4).astype(np.float32)
        if L > 3:
            q[1, 3] = np.nan
            q[2, 0] = np.inf
            q[3, 7] = 3e38   # 2q overflows to inf
        nb = check_neighbors(q, K)
        if L > 3:
            assert np.all(nb["slot"][1:4] == -1)


def test_neighbors_workload_queries():
    for name in ("k4-m32-f32-uniform", "k4-m32-f32-gmm64"):
        w = W.WORKLOADS[name]
        _say("neighbors workload", name)
        check_neighbors(W.queries(w).reshape(-1, 8), w.K)
    for name in ("k8-m64-f32-uniform", "k12-m64-bf16-proj", "k14-m32-bf16-zipf"):
        w = W.WORKLOADS[name]
        _say("neighbors workload sample", name)
        q = W.queries(w).reshape(-1, 8)
        idx = np.random.default_rng(1).choice(q.shape[0], 6000, replace=False)
        check_neighbors(q[idx], w.K)


def test_empty_batch_is_noop():
    q = torch.empty((0, 4, 8), dtype=torch.float32, device=DEV)
    slot, w, d2 = lram.neighbors(q, (4,) * 8)
    table = torch.zeros((4 ** 8, 32), device=DEV)
    out = lram.forward(q, table, (4,) * 8)
    assert out.shape == (0, 4, 32)
    g = torch.empty((0, 4, 32), device=DEV)
    gt, gq = lram.backward(q, table, (4,) * 8, g)
    torch.cuda.synchronize()
    assert gt.abs().sum().item() == 0


def _small_table(K, m, dtype, seed=0):
    N = int(np.prod(K))
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    t = torch.randn((N, m), generator=g, device=DEV) * 0.02
    return t.to(dtype)


def _tol(dtype):
    return 1e-5 if dtype == torch.float32 else 2e-2


@pytest.mark.parametrize("mode", ["atomic", "sorted", "merged"])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("m", [32, 64])
@pytest.mark.parametrize("K", [(4,) * 8, (2, 4, 6, 8, 2, 4, 6, 8)])
def test_forward_backward_small(K, m, dtype, mode):
    _say("fwd/bwd K=%s m=%d %s %s" % (K, m, dtype, mode))
    rng = np.random.default_rng(11)
    L = 3000
    q_np = (rng.random((L, 8)) * np.asarray(K)).astype(np.float32)
    q_np[:10] = special_queries(K)[:10]
    q_np[10, 2] = np.nan
    q = torch.from_numpy(q_np).to(DEV)
    table = _small_table(K, m, dtype)
    G = torch.randn((L, m), device=DEV, dtype=torch.float32)
    out = lram.forward(q, table, K)
    gt, gq = lram.backward(q, table, K, G, mode=mode)
    torch.cuda.synchronize()
    nb = oracle.neighbors(q_np, K)
    tab = table.float().cpu().numpy()
    rows = oracle.gather_rows(tab, nb["slot"])
    ref = oracle.forward(nb, rows)
    err = _rel_rows(out.float().cpu().numpy(), ref)
    assert err.max() <= _tol(dtype), err.max()
    # dq: the fp32 kernel vs fp64 oracle
    Gn = G.cpu().numpy()
    dq_ref = oracle.grad_query(nb, rows, Gn)
    err = _rel_rows(gq.cpu().numpy(), dq_ref)
    assert err.max() <= 1e-5, err.max()
    dV_ref = oracle.grad_table_dense(nb, Gn, int(np.prod(K)))
    dV = gt.cpu().numpy()
    touched = np.unique(nb["slot"][nb["slot"] >= 0])
    err = _rel_rows(dV[touched], dV_ref[touched])
    assert err.max() <= 1e-5, err.max()
    untouched = np.setdiff1d(np.arange(dV.shape[0]), touched)
    assert np.all(dV[untouched] == 0)
    assert np.all(out.float().cpu().numpy()[10] == 0) and np.all(gq.cpu().numpy()[10] == 0)


@pytest.mark.parametrize("mode", ["atomic", "sorted", "merged"])
def test_backward_accumulates(mode):
    K = (4,) * 8
    rng = np.random.default_rng(12)
    q = torch.from_numpy((rng.random((500, 8)) * 4).astype(np.float32)).to(DEV)
    table = _small_table(K, 32, torch.float32)
    G = torch.randn((500, 32), device=DEV)
    gt1, gq1 = lram.backward(q, table, K, G, mode=mode)
    gt2 = gt1.clone()
    lram.backward(q, table, K, G, grad_table=gt2, want_grad_q=False, mode=mode)
    # dq alone (no value gradient) is the same in every mode
    _, gq3 = lram.backward(q, table, K, G, grad_table=False, mode=mode)
    torch.cuda.synchronize()
    assert torch.equal(gq1, gq3)
    # atomic accumulation order varies between calls: compare at the fp32 parity bar
    np.testing.assert_allclose(gt2.cpu().numpy(), 2 * gt1.cpu().numpy(), rtol=1e-5, atol=1e-7)


@pytest.mark.parametrize("mode", ["atomic", "sorted", "merged"])
@pytest.mark.parametrize("name", ["k4-m32-f32-uniform", "k4-m32-f32-gmm64"])
def test_workload_full_parity(name, mode):
    """Small workloads in full: every lookup, every output."""
    w = W.WORKLOADS[name]
    _say("full parity", name, mode)
    q_np = W.queries(w)
    q = torch.from_numpy(q_np).to(DEV)
    table = W.make_table(w, DEV)
    G = W.grad_out(w, DEV)
    out = lram.forward(q, table, w.K)
    gt, gq = lram.backward(q, table, w.K, G, mode=mode)
    torch.cuda.synchronize()
    nb = oracle.neighbors(q_np, w.K)
    rows = oracle.gather_rows(table.float().cpu().numpy(), nb["slot"])
    assert _rel_rows(out.cpu().numpy().reshape(w.L, -1), oracle.forward(nb, rows).reshape(w.L, -1)).max() <= 1e-5
    Gn = G.cpu().numpy()
    dq_ref = oracle.grad_query(nb, rows, Gn)
    assert _rel_rows(gq.cpu().numpy().reshape(w.L, -1), dq_ref.reshape(w.L, -1)).max() <= 1e-5
    uniq, acc = oracle.grad_table_rows(nb, Gn)
    dV = gt.cpu().numpy()
    assert _rel_rows(dV[uniq], acc).max() <= 1e-5
    mask = np.ones(w.N, bool)
    mask[uniq] = False
    assert np.all(dV[mask] == 0)


@pytest.mark.parametrize("mode", ["atomic", "sorted", "merged"])
def test_hot_rows(mode):
    """Many lookups on a few lattice cells: runs of one location span many
    64-pair chunks of the sorted reduction (and contend in the atomic one)."""
    _say("hot rows", mode)
    K = (8,) * 8
    rng = np.random.default_rng(13)
    centres = (rng.random((3, 8)) * 8)
    L = 70001  # enough lookups for full 64-lookup merge batches, and a ragged last one
    q_np = (centres[rng.integers(0, 3, L)] + 0.05 * rng.standard_normal((L, 8))).astype(np.float32)
    q = torch.from_numpy(q_np).to(DEV)
    table = _small_table(K, 32, torch.float32)
    G = torch.randn((L, 32), device=DEV)
    gt, gq = lram.backward(q, table, K, G, mode=mode)
    torch.cuda.synchronize()
    nb = oracle.neighbors(q_np, K)
    uniq, acc = oracle.grad_table_rows(nb, G.cpu().numpy())
    dV = gt.cpu().numpy()
    assert uniq.size < 600
    assert _rel_rows(dV[uniq], acc).max() <= 1e-5
    mask = np.ones(dV.shape[0], bool)
    mask[uniq] = False
    assert np.all(dV[mask] == 0)
    rows = oracle.gather_rows(table.cpu().numpy(), nb["slot"])
    assert _rel_rows(gq.cpu().numpy(), oracle.grad_query(nb, rows, G.cpu().numpy())).max() <= 1e-5


def test_mixed_batches_merged():
    """Merged scatter on a batch whose sorted order holds both clustered runs
    (merged in LDS) and thinly spread lookups (direct atomics), with full
    64-lookup batches and a ragged last one."""
    _say("mixed batches merged")
    K = (8,) * 8
    rng = np.random.default_rng(14)
    centres = rng.random((5, 8)) * 8
    L = 90003
    q_np = (rng.random((L, 8)) * 8).astype(np.float32)
    hot = rng.random(L) < 0.5
    q_np[hot] = np.mod(centres[rng.integers(0, 5, hot.sum())] + 0.2 * rng.standard_normal((hot.sum(), 8)),
                       8).astype(np.float32)
    q = torch.from_numpy(q_np).to(DEV)
    table = _small_table(K, 32, torch.bfloat16)
    G = torch.randn((L, 32), device=DEV)
    gt, gq = lram.backward(q, table, K, G, mode="merged")
    gta, gqa = lram.backward(q, table, K, G, mode="atomic")
    torch.cuda.synchronize()
    assert torch.equal(gq, gqa)  # dq does not depend on the scatter
    nb = oracle.neighbors(q_np, K)
    uniq, acc = oracle.grad_table_rows(nb, G.cpu().numpy())
    dV = gt.cpu().numpy()
    assert _rel_rows(dV[uniq], acc).max() <= 1e-5
    mask = np.ones(dV.shape[0], bool)
    mask[uniq] = False
    assert np.all(dV[mask] == 0)


def test_merged_batches_near_capacity():
    """Merged scatter on batches whose lookups are mostly spread thinly but
    share their closest lattice point often enough (two in five) for the merge
    to run: about 1,600 distinct locations among a batch's 2,048 pairs, so the
    group locations compacted over the hash tags and the pair weights in the
    tags' upper half nearly fill their halves; three full batches and a ragged one."""
    _say("merged batches near capacity")
    K = (8,) * 8
    rng = np.random.default_rng(21)
    npair, nsingle = 42, 127
    base = rng.random((npair, 8)) * 8
    twins = np.mod(base + 1e-3 * rng.standard_normal((npair, 8)), 8)
    q_np = np.concatenate([base, twins, rng.random((nsingle, 8)) * 8]).astype(np.float32)
    q_np = q_np[rng.permutation(q_np.shape[0])]
    L = q_np.shape[0]
    assert L == 3 * 64 + 19
    q = torch.from_numpy(q_np).to(DEV)
    table = _small_table(K, 32, torch.float32)
    G = torch.randn((L, 32), device=DEV)
    gt, gq = lram.backward(q, table, K, G, mode="merged")
    gta, gqa = lram.backward(q, table, K, G, mode="atomic")
    torch.cuda.synchronize()
    assert torch.equal(gq, gqa)
    nb = oracle.neighbors(q_np, K)
    cells = nb["slot"][:, 0]
    assert np.unique(cells).size <= L - npair + 2  # the twins share their cell
    uniq, acc = oracle.grad_table_rows(nb, G.cpu().numpy())
    assert uniq.size > 0.75 * 32 * L
    dV = gt.cpu().numpy()
    assert _rel_rows(dV[uniq], acc).max() <= 1e-5
    mask = np.ones(dV.shape[0], bool)
    mask[uniq] = False
    assert np.all(dV[mask] == 0)
    assert _rel_rows(dV[uniq], gta.cpu().numpy()[uniq]).max() <= 1e-5


@pytest.mark.parametrize("mode", ["sorted", "merged"])
def test_workspace_errors(mode):
    K = (4,) * 8
    q = torch.rand((100, 8), device=DEV) * 4
    table = _small_table(K, 32, torch.float32)
    G = torch.randn((100, 32), device=DEV)
    need = lram.backward_workspace_bytes(100, 1, 32, mode)
    assert need > 100 * 24
    small = torch.empty(need - 256, dtype=torch.uint8, device=DEV)
    with pytest.raises(lram.LramError):
        lram.backward(q, table, K, G, mode=mode, workspace=small)


def test_binding_rejects_mismatched_buffers():
    """The C ABI sees raw pointers only; the binding checks the shape, dtype and
    device of every buffer before a kernel could run past its end."""
    K = (4,) * 8
    N = 4 ** 8
    q = torch.rand((100, 8), device=DEV) * 4
    z = torch.randn((100, 16), device=DEV)
    table = _small_table(K, 32, torch.float32)
    G = torch.randn((100, 32), device=DEV)
    f32 = dict(dtype=torch.float32, device=DEV)
    bad = [
        lambda: lram.forward(q, table, K, out=torch.empty((99, 32), **f32)),
        lambda: lram.forward(q, table, K, out=torch.empty((100, 64), **f32)),
        lambda: lram.forward(q, table.cpu(), K),
        lambda: lram.forward(q, table.reshape(-1), K),
        lambda: lram.backward(q, table, K, torch.randn((100, 16), **f32)),
        lambda: lram.backward(q, table, K, G, grad_table=torch.zeros((N - 1, 32), **f32)),
        lambda: lram.backward(q, table, K, G, grad_q=torch.empty((100, 4), **f32)),
        lambda: lram.backward(q, table, K, G, k=16, grad_table=torch.zeros((N, 16), **f32)),
        lambda: lram.theta_forward(z, table, K, out=torch.empty((100, 16), **f32)),
        lambda: lram.theta_backward(z, table, K, G, grad_z=torch.empty((100, 8), **f32)),
        lambda: lram.access_histogram(q, K, hist=torch.zeros(N // 2, **f32)),
        lambda: lram.access_stats(torch.zeros((N, 1), **f32)),
        lambda: lram.sparse_adam(table, torch.zeros((N, 16), **f32), torch.zeros((N, 32), **f32),
                                 torch.zeros((N, 32), **f32), 1),
    ]
    for i, call in enumerate(bad):
        with pytest.raises(lram.LramError):
            call()
            pytest.fail("case %d accepted" % i)
    torch.cuda.synchronize()


def test_lookup_autograd_matches_abi():
    """The autograd wrapper gives the ABI's output and gradients, also for a
    non-contiguous query view."""
    K = (4,) * 8
    rng = np.random.default_rng(31)
    q = torch.from_numpy((rng.random((8, 300)) * 4).astype(np.float32)).to(DEV).t()   # [300, 8] view
    assert not q.is_contiguous()
    table = _small_table(K, 32, torch.float32)
    G = torch.randn((300, 32), device=DEV)
    qr = q.clone().requires_grad_(True)
    tr = table.clone().requires_grad_(True)
    out = lram.lookup(qr, tr, K)
    (out * G).sum().backward()
    ref = lram.forward(q.contiguous(), table, K)
    gt, gq = lram.backward(q.contiguous(), table, K, G)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), ref)
    assert torch.equal(qr.grad, gq)
    np.testing.assert_allclose(tr.grad.cpu().numpy(), gt.cpu().numpy(), rtol=1e-5, atol=1e-7)
