"""The neighbour lists the forward saves (Sec. 2.6: the indices and weights
handed to the autograd wrapper) and the backward that reuses them.

  * saved lists: per lookup the same (location, weight) entries as
    lram_neighbors, bit-exact, padding last;
  * backward with the lists: dq bit-identical to the backward that searches
    again, the value gradient bit-identical under the (reproducible) sorted
    scatter and within 1e-5 per row under the atomic and merged ones;
  * entries whose location lies outside [0, N) act as padding;
  * the autograd wrapper with save_lists gives the same gradients.
"""
import numpy as np
import pytest
import torch

import paper_2107_03474_amd as lram
from test_gpu_parity import _rel_rows, special_queries

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _say(*a):
    print(*a, flush=True)


def _setup(K, L, m, dtype, seed, clustered=False):
    rng = np.random.default_rng(seed)
    Kf = np.asarray(K, np.float64)
    q_np = rng.random((L, 8)) * Kf
    if clustered:
        c = rng.random((30, 8)) * Kf
        hot = rng.random(L) < 0.7
        q_np[hot] = np.mod(c[rng.integers(0, 30, hot.sum())] + 0.3 * rng.standard_normal((hot.sum(), 8)), Kf)
    q_np = q_np.astype(np.float32)
    sp = special_queries(K)
    n = min(L, 64)
    for t in range(n):
        q_np[(64 * t + t) % L] = sp[t % sp.shape[0]]
    q_np[min(L - 1, 5), 1] = np.nan
    q = torch.from_numpy(q_np).to(DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    N = int(np.prod(K))
    table = (torch.randn((N, m), generator=g, device=DEV) * 0.02).to(dtype)
    G = torch.randn((L, m), generator=g, device=DEV)
    return q, table, G


@pytest.mark.parametrize("K,L", [((4,) * 8, 4096), ((8,) * 8, 300000), ((2, 4, 6, 8, 2, 4, 6, 8), 3001)])
def test_saved_lists_are_the_neighbour_lists(K, L):
    _say("saved lists K=%s L=%d" % (K, L))
    q, table, _ = _setup(K, L, 32, torch.float32, 1)
    nl = lram.new_lists(q)
    out = lram.forward(q, table, K, lists=nl)
    ref = lram.forward(q, table, K)
    slot, w, _ = lram.neighbors(q, K, want_d2=False)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    s_saved, w_saved = nl.slot.cpu().numpy(), nl.w.cpu().numpy()
    s_ref, w_ref = slot.cpu().numpy(), w.cpu().numpy()
    cnt = (s_saved >= 0).sum(1)
    assert np.array_equal(cnt, (s_ref >= 0).sum(1))
    assert np.all((s_saved >= 0) == (np.arange(32)[None, :] < cnt[:, None]))   # padding last
    assert np.all(w_saved[s_saved < 0] == 0) and np.all(nl.code.cpu().numpy()[s_saved < 0] == 0)
    # same entries: sort both by (location, weight bits)
    def canon(s, w):
        key = s.astype(np.int64) * (1 << 32) + w.view(np.uint32).astype(np.int64)
        return np.sort(key, axis=1)
    assert np.array_equal(canon(s_saved, w_saved), canon(s_ref, w_ref))


@pytest.mark.parametrize("mode", ["atomic", "sorted", "merged"])
@pytest.mark.parametrize("K,L,dtype", [((4,) * 8, 4096, torch.float32), ((8,) * 8, 262144, torch.bfloat16)])
def test_backward_with_saved_lists(K, L, dtype, mode):
    _say("backward with saved lists K=%s L=%d %s" % (K, L, mode))
    q, table, G = _setup(K, L, 32, dtype, 2, clustered=True)
    nl = lram.new_lists(q)
    lram.forward(q, table, K, lists=nl)
    gt, gq = lram.backward(q, table, K, G, mode=mode, lists=nl)
    gt_ref, gq_ref = lram.backward(q, table, K, G, mode=mode)
    torch.cuda.synchronize()
    assert torch.equal(gq, gq_ref)
    touched = (gt_ref != 0).any(1)
    assert torch.equal((gt != 0).any(1), touched)
    if mode == "sorted":
        assert torch.equal(gt, gt_ref)
    else:
        assert _rel_rows(gt[touched].cpu().numpy(), gt_ref[touched].cpu().numpy()).max() <= 1e-5


def test_saved_list_entries_outside_the_table_are_padding():
    K = (4,) * 8
    N = 4 ** 8
    q, table, G = _setup(K, 2000, 32, torch.float32, 3)
    nl = lram.new_lists(q)
    lram.forward(q, table, K, lists=nl)
    bad = lram.Lists(nl.slot.clone(), nl.w.clone(), nl.code.clone())
    pad = lram.Lists(nl.slot.clone(), nl.w.clone(), nl.code.clone())
    rows = torch.arange(0, 2000, 7, device=DEV)
    bad.slot[rows, 3] = N + 5
    bad.slot[rows, 9] = 2 ** 31 - 1
    pad.slot[rows, 3] = -1
    pad.slot[rows, 9] = -1
    gt_b, gq_b = lram.backward(q, table, K, G, mode="sorted", lists=bad)
    gt_p, gq_p = lram.backward(q, table, K, G, mode="sorted", lists=pad)
    torch.cuda.synchronize()
    assert torch.equal(gq_b, gq_p) and torch.equal(gt_b, gt_p)


def test_autograd_with_saved_lists():
    K = (4,) * 8
    q, table, G = _setup(K, 3000, 32, torch.float32, 4)
    grads = []
    for save in (False, True):
        qr = q.clone().requires_grad_(True)
        tr = table.clone().requires_grad_(True)
        out = lram.lookup(qr, tr, K, mode="sorted", save_lists=save)
        (out * G).sum().backward()
        grads.append((out.detach(), qr.grad, tr.grad))
    torch.cuda.synchronize()
    for a, b in zip(*grads):
        assert torch.equal(a, b)
