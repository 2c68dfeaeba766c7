"""GPU parity of the lookup order (lram_order) and of the forward and
backward calls that take it.

  * keys: bit-exact -- the location of the lookup's closest lattice point as
    the oracle enumerates it (where two points are equally close in exact
    arithmetic, the key is one of them: the fp32 recipe may separate such a
    tie by an ulp), N for a non-finite query; keys sorted,
    positions a permutation, equal keys in lookup order (the sort is stable);
    the gate count equals the number of positions whose key equals a
    neighbour's; the sort's failure word is 0;
  * the same points given as q - K and q + 3K (exact in fp32 on a 2^-10 grid)
    give the same keys, positions and gate count, and the merged backward the
    same gradients (Sec. 2.2: the torus periods);
  * forward with an order: bit-identical to the forward without one (each
    lookup's arithmetic does not depend on where it runs); backward with an
    order: dq bit-identical, value-gradient rows within 1e-5 of the oracle;
  * an order whose positions name lookups outside [0, L) skips them.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2107_03474_amd as lram
from test_gpu_parity import _rel_rows, special_queries

pytestmark = pytest.mark.gpu
DEV = "cuda"
K8 = (8,) * 8


def _say(*a):
    print(*a, flush=True)


def _clustered(L, seed, K=K8, ncent=50, sigma=0.3, grid=None):
    rng = np.random.default_rng(seed)
    Kf = np.asarray(K, np.float64)
    q = rng.random((L, 8)) * Kf
    hot = rng.random(L) < 0.7
    centres = rng.random((ncent, 8)) * Kf
    q[hot] = np.mod(centres[rng.integers(0, ncent, hot.sum())] + sigma * rng.standard_normal((hot.sum(), 8)), Kf)
    if grid:
        q = np.mod(np.floor(q * grid) / grid, Kf)
    return q.astype(np.float32)


def _view(buf, L):
    cnt, keys, perm = lram.order_view(buf, L)
    return int(cnt.item()), keys.cpu().numpy().astype(np.int64), perm.cpu().numpy().astype(np.int64)


def _check_order(q_np, K, buf):
    L = q_np.shape[0]
    N = int(np.prod(K))
    cnt, keys, perm = _view(buf, L)
    assert int(buf[4:8].view(torch.int32).item()) == 0      # the sort's failure word
    assert np.all(np.diff(keys) >= 0)
    assert np.array_equal(np.sort(perm), np.arange(L))
    same = np.diff(keys) == 0
    assert np.all(np.diff(perm)[same] > 0)                     # stable
    shared = np.zeros(L, bool)
    shared[1:] |= same
    shared[:-1] |= same
    assert cnt == int(shared.sum())
    key_of = np.empty(L, np.int64)
    key_of[perm] = keys
    nb = oracle.neighbors(q_np, K)
    finite = np.all(np.isfinite(q_np), axis=1)
    assert np.all(key_of[~finite] == N)
    # the decoder finds a closest point in exact arithmetic; where two points
    # are equally close there, the fp32 recipe that orders the oracle's list
    # may separate them by an ulp and list the other one first
    first = key_of == nb["slot"][:, 0]
    near = nb["d2"] <= nb["d2"][:, :1] * np.float32(1 + 2 ** -20)
    for l in np.nonzero(finite & ~first)[0]:
        assert key_of[l] in nb["slot"][l][near[l]], l
    tied = nb["d2"][:, 0] == nb["d2"][:, 1]
    assert (finite & ~first & ~tied).sum() <= max(2, L // 10000)
    return cnt, keys, perm


@pytest.mark.parametrize("K", [K8, (2, 4, 6, 8, 10, 2, 4, 6), (14,) * 8])
def test_order_keys_and_positions(K):
    _say("order K=%s" % (K,))
    q_np = _clustered(40000, 1, K=K)
    sp = special_queries(K)
    q_np[:sp.shape[0]] = sp
    q_np[100, 3] = np.nan
    q_np[101, 0] = np.inf
    q = torch.from_numpy(q_np).to(DEV)
    buf = lram.order(q, K)
    torch.cuda.synchronize()
    cnt, _, _ = _check_order(q_np, K, buf)
    assert cnt > 1000


def test_order_ragged_sizes():
    rng = np.random.default_rng(2)
    for L in (1, 2, 255, 4097, 70001):
        q_np = (rng.random((L, 8)) * 8).astype(np.float32)
        q = torch.from_numpy(q_np).to(DEV)
        buf = lram.order(q, K8)
        torch.cuda.synchronize()
        _check_order(q_np, K8, buf)


def test_order_several_lookback_groups():
    """Sizes whose tiles (4,096 lookups) span several look-back groups of 32
    tiles, with a ragged last tile and group: 300,007 lookups against the
    oracle; 4,194,309 (33 groups, as at the billion-location workload plus a
    ragged tile) on sort properties and against the closest points that
    lram_neighbors lists first."""
    rng = np.random.default_rng(7)
    q_np = _clustered(300007, 3)
    q_np[5] = np.nan
    q = torch.from_numpy(q_np).to(DEV)
    buf = lram.order(q, K8)
    torch.cuda.synchronize()
    _check_order(q_np, K8, buf)
    K = (14,) * 8
    L = 4194309
    q_np = (rng.random((L, 8)) * 14).astype(np.float32)
    centres = rng.random((2000, 8)) * 14               # half the lookups around 2,000 points: shared cells
    q_np[: L // 2] = np.mod(centres[rng.integers(0, 2000, L // 2)] + 0.02 * rng.standard_normal((L // 2, 8)),
                            14).astype(np.float32)
    q = torch.from_numpy(q_np).to(DEV)
    buf = lram.order(q, K)
    slot, _, d2 = lram.neighbors(q, K)
    torch.cuda.synchronize()
    assert int(buf[4:8].view(torch.int32).item()) == 0
    cnt, keys, perm = _view(buf, L)
    assert np.all(np.diff(keys) >= 0)
    assert np.array_equal(np.sort(perm), np.arange(L))
    same = np.diff(keys) == 0
    assert np.all(np.diff(perm)[same] > 0)
    shared = np.zeros(L, bool)
    shared[1:] |= same
    shared[:-1] |= same
    assert cnt == int(shared.sum()) and cnt > L // 4
    key_of = np.empty(L, np.int64)
    key_of[perm] = keys
    s0 = slot[:, 0].cpu().numpy()
    off = np.nonzero(key_of != s0)[0]
    if off.size:
        sl, dd = slot[off].cpu().numpy(), d2[off].cpu().numpy()
        near = dd <= dd[:, :1] * np.float32(1 + 2 ** -20)
        assert np.all(((sl == key_of[off][:, None]) & near).any(axis=1))
        assert int((dd[:, 0] != dd[:, 1]).sum()) <= max(2, L // 10000)


def test_order_and_merged_backward_see_through_the_wrap():
    """The merge gate and the merged backward do not depend on which copy of a
    torus point the caller passes (negative queries, queries past K)."""
    _say("order wrap")
    L = 140000
    q_np = _clustered(L, 3, grid=1024)
    Kf = np.asarray(K8, np.float32)
    g = torch.Generator(device=DEV)
    g.manual_seed(5)
    table = torch.randn((8 ** 8, 32), generator=g, device=DEV) * 0.02
    G = torch.randn((L, 32), generator=g, device=DEV)
    res = []
    for shift in (0.0, -1.0, 3.0):
        qs = (q_np + shift * Kf).astype(np.float32)
        assert np.array_equal(qs - np.float32(shift) * Kf, q_np)  # exact on the grid
        q = torch.from_numpy(qs).to(DEV)
        ws = torch.empty(lram.backward_workspace_bytes(L, 1, 32, "merged"), dtype=torch.uint8, device=DEV)
        gt, gq = lram.backward(q, table, K8, G, mode="merged", workspace=ws)
        ordbuf = lram.order(q, K8)
        torch.cuda.synchronize()
        res.append((_view(ws, L), _view(ordbuf, L), gt, gq))
    (c0, k0, p0), _, gt0, gq0 = res[0]
    assert c0 > L // 2
    for (c, k, p), (co, ko, po), gt, gq in res:
        assert c == c0 and co == c0
        assert np.array_equal(k, k0) and np.array_equal(ko, k0)
        assert np.array_equal(p, p0) and np.array_equal(po, p0)
        assert torch.equal(gq, gq0)
        touched = (gt0 != 0).any(1)
        assert torch.equal((gt != 0).any(1), touched)
        assert _rel_rows(gt[touched].cpu().numpy(), gt0[touched].cpu().numpy()).max() <= 1e-5


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_forward_with_order_is_identical(dtype):
    _say("forward with order", dtype)
    L = 300000
    q_np = _clustered(L, 4)
    sp = special_queries(K8)
    for t in range(64):  # special queries at every position of a 64-lookup wave
        q_np[64 * (97 + t) + t] = sp[t % sp.shape[0]]
    q_np[1234, 5] = np.nan
    q = torch.from_numpy(q_np).to(DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(6)
    table = (torch.randn((8 ** 8, 64), generator=g, device=DEV) * 0.02).to(dtype)
    ref = lram.forward(q, table, K8)
    buf = lram.order(q, K8)
    out = lram.forward(q, table, K8, order=buf)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


@pytest.mark.parametrize("mode", ["atomic", "merged"])
def test_backward_with_order(mode):
    _say("backward with order", mode)
    L = 200003
    q_np = _clustered(L, 7)
    q_np[17, 2] = np.inf
    q = torch.from_numpy(q_np).to(DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(8)
    table = (torch.randn((8 ** 8, 32), generator=g, device=DEV) * 0.02).to(torch.bfloat16)
    G = torch.randn((L, 32), generator=g, device=DEV)
    buf = lram.order(q, K8)
    gt, gq = lram.backward(q, table, K8, G, mode=mode, order=buf)
    _, gq_ref = lram.backward(q, table, K8, G, mode=mode, grad_table=False)
    torch.cuda.synchronize()
    assert torch.equal(gq, gq_ref)
    nb = oracle.neighbors(q_np, K8)
    uniq, acc = oracle.grad_table_rows(nb, G.cpu().numpy())
    dV = gt.cpu().numpy()
    assert _rel_rows(dV[uniq], acc).max() <= 1e-5
    mask = np.ones(dV.shape[0], bool)
    mask[uniq] = False
    assert np.all(dV[mask] == 0)


def test_positions_outside_the_batch_are_skipped():
    """An order naming lookups that do not exist: those positions do nothing,
    the others run as usual."""
    L = 5000
    rng = np.random.default_rng(9)
    q_np = (rng.random((L, 8)) * 8).astype(np.float32)
    q = torch.from_numpy(q_np).to(DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(10)
    table = torch.randn((8 ** 8, 32), generator=g, device=DEV) * 0.02
    G = torch.randn((L, 32), generator=g, device=DEV)
    buf = lram.order(q, K8)
    _, _, perm = lram.order_view(buf, L)
    perm.copy_(torch.arange(L, dtype=torch.int32, device=DEV))
    perm[10:20] = -1                          # 0xFFFFFFFF: beyond any lookup
    out = torch.full((L, 32), 7.0, device=DEV)
    lram.forward(q, table, K8, out=out, order=buf)
    gq = torch.full((L, 8), 7.0, device=DEV)
    gt, _ = lram.backward(q, table, K8, G, mode="atomic", order=buf, grad_q=gq)
    ref = lram.forward(q, table, K8)
    _, gq_ref = lram.backward(q, table, K8, G, mode="atomic", grad_table=False)
    torch.cuda.synchronize()
    keep = torch.ones(L, dtype=torch.bool, device=DEV)
    keep[10:20] = False
    assert torch.all(out[10:20] == 7.0) and torch.all(gq[10:20] == 7.0)
    assert torch.equal(out[keep], ref[keep]) and torch.equal(gq[keep], gq_ref[keep])
    sel = np.r_[0:10, 20:L]
    nb = oracle.neighbors(q_np[sel], K8)
    uniq, acc = oracle.grad_table_rows(nb, G.cpu().numpy()[sel])
    dV = gt.cpu().numpy()
    assert _rel_rows(dV[uniq], acc).max() <= 1e-5
    mask = np.ones(dV.shape[0], bool)
    mask[uniq] = False
    assert np.all(dV[mask] == 0)
