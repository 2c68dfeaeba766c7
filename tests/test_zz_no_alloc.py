"""lram_backward_noalloc (the backward whose scatter workspace is the
library's static per-GPU array) against lram_backward with a caller-owned
workspace, through the C ABI: two calls in a row on the same GPU, the second
smaller, so the array keeps the first call's contents when the second starts.

  * sorted scatter: both sides are bit-reproducible, so grad_table and grad_q
    must be bit-identical;
  * merged scatter: grad_q bit-identical (it does not depend on the scatter),
    grad_table rows within the fp32 parity bar (1e-5 per row, relative L2),
    whose atomics add in a varying order; untouched rows exactly 0;
  * a call whose workspace would not fit the array is refused on the host.
"""
import numpy as np
import pytest
import torch

import paper_2107_03474_amd as lram

pytestmark = pytest.mark.gpu
DEV = "cuda"
K = (8,) * 8


def _say(*a):
    print(*a, flush=True)


def _inputs(L, seed, m=32):
    rng = np.random.default_rng(seed)
    centres = rng.random((40, 8)) * 8
    q = rng.random((L, 8)) * 8
    hot = rng.random(L) < 0.6
    q[hot] = np.mod(centres[rng.integers(0, 40, hot.sum())] + 0.3 * rng.standard_normal((hot.sum(), 8)), 8)
    q = torch.from_numpy(q.astype(np.float32)).to(DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    G = torch.randn((L, m), generator=g, device=DEV)
    return q, G


def _rel_rows(a, b):
    num = (a - b).double().norm(dim=1)
    den = b.double().norm(dim=1)
    return torch.where(den > 0, num / den.clamp(min=1e-300), num)


@pytest.mark.parametrize("mode,sizes", [("sorted", (60000, 20001)), ("merged", (300000, 131077))])
def test_noalloc_matches_backward(mode, sizes):
    N = 8 ** 8
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    table = (torch.randn((N, 32), generator=g, device=DEV) * 0.02).to(torch.bfloat16)
    for call, L in enumerate(sizes):
        _say("noalloc %s call %d: %d lookups" % (mode, call, L))
        q, G = _inputs(L, 10 + call)
        gt_ref = torch.zeros((N, 32), device=DEV)
        gq_ref = torch.empty((L, 8), device=DEV)
        lram.backward(q, table, K, G, grad_table=gt_ref, grad_q=gq_ref, mode=mode)
        gt = torch.zeros((N, 32), device=DEV)
        gq = torch.empty((L, 8), device=DEV)
        lram.backward_noalloc(q, table, K, G, gt, gq, mode=mode)
        torch.cuda.synchronize()
        assert torch.equal(gq, gq_ref)
        touched = (gt_ref != 0).any(1)
        assert int(touched.sum()) > 1000
        if mode == "sorted":
            assert torch.equal(gt, gt_ref)
        else:
            assert _rel_rows(gt[touched], gt_ref[touched]).max().item() <= 1e-5
            assert torch.count_nonzero(gt[~touched]).item() == 0
        del gt_ref, gq_ref, gt, gq


def test_noalloc_refuses_what_does_not_fit():
    q = torch.zeros((200000, 8), device=DEV)
    table = torch.zeros((8 ** 8, 32), device=DEV)
    G = torch.zeros((200000, 32), device=DEV)
    gt = torch.zeros((8 ** 8, 32), device=DEV)
    with pytest.raises(lram.LramError, match="workspace"):
        lram.backward_noalloc(q, table, K, G, gt, mode="sorted")   # 32 x 200000 pairs do not fit
    torch.cuda.synchronize()
    assert torch.count_nonzero(gt).item() == 0
