"""Stream and graph behaviour of the C ABI.

* Every kernel of a call is enqueued on the stream the caller names: the same
  calls on a side stream give the default stream's results.
* A forward + backward step, in each scatter mode, can be captured into a HIP
  graph and replayed: a call allocates nothing, never synchronises with the
  host and clears its own counters with a kernel (no memset node).  Each
  replay, with eager work and synchronisations in between, reproduces the
  eager step.

Bars: forward output and dq bit-identical (each lookup is reduced by one wave
in a fixed order); the value gradient, whose atomics land in any order, per
touched row within 1e-5 relative L2, and untouched rows exactly 0.
"""
import numpy as np
import pytest
import torch

import paper_2107_03474_amd as lram

pytestmark = pytest.mark.gpu
DEV = "cuda"
K = (6,) * 8
MODES = ["atomic", "sorted", "merged"]


def _say(*a):
    print(*a, flush=True)


def _inputs(L=20000, m=32, seed=3):
    """Half the queries around 64 centres (so the merged scatter merges), half uniform."""
    rng = np.random.default_rng(seed)
    centres = rng.random((64, 8)) * 6
    qc = centres[rng.integers(0, 64, L // 2)] + 0.3 * rng.standard_normal((L // 2, 8))
    qu = rng.random((L - L // 2, 8)) * 6
    q = np.concatenate([qc, qu]).astype(np.float32)
    G = rng.standard_normal((L, m)).astype(np.float32)
    gen = torch.Generator(device=DEV).manual_seed(seed)
    table = (torch.randn((int(np.prod(K)), m), generator=gen, device=DEV) * 0.02).to(torch.bfloat16)
    return torch.from_numpy(q).to(DEV), table, torch.from_numpy(G).to(DEV)


def _check_grad_table(gt, ref):
    a = gt.double().cpu().numpy()
    b = ref.double().cpu().numpy()
    touched = np.any(b != 0, axis=1)
    assert np.array_equal(np.any(a != 0, axis=1), touched)
    num = np.linalg.norm(a[touched] - b[touched], axis=1)
    den = np.linalg.norm(b[touched], axis=1)
    assert np.max(num / den) <= 1e-5


@pytest.mark.parametrize("mode", MODES)
def test_side_stream_matches_default(mode):
    _say("side stream, scatter %s" % mode)
    q, table, G = _inputs()
    out0 = lram.forward(q, table, K)
    gt0, gq0 = lram.backward(q, table, K, G, mode=mode)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out1 = lram.forward(q, table, K)
        gt1, gq1 = lram.backward(q, table, K, G, mode=mode)
    s.synchronize()
    assert torch.equal(out0, out1)
    assert torch.equal(gq0, gq1)
    _check_grad_table(gt1, gt0)


@pytest.mark.parametrize("mode", MODES)
def test_graph_capture_replays(mode):
    _say("graph capture, scatter %s" % mode)
    q, table, G = _inputs(seed=4)
    N, m = table.shape
    L = q.shape[0]
    out = torch.empty((L, m), dtype=table.dtype, device=DEV)
    gq = torch.empty((L, 8), dtype=torch.float32, device=DEV)
    gt = torch.zeros((N, m), dtype=torch.float32, device=DEV)
    nws = lram.backward_workspace_bytes(L, 1, m, mode)
    ws = torch.empty(nws, dtype=torch.uint8, device=DEV) if nws else None

    def step():
        gt.zero_()
        lram.forward(q, table, K, out=out)
        lram.backward(q, table, K, G, grad_table=gt, grad_q=gq, mode=mode, workspace=ws)

    step()
    torch.cuda.synchronize()
    ref_out, ref_gq, ref_gt = out.clone(), gq.clone(), gt.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for r in range(3):
        out.fill_(0)
        gq.fill_(0)
        gt.fill_(1.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        _say("  replay %d" % r)
        assert torch.equal(out, ref_out)
        assert torch.equal(gq, ref_gq)
        _check_grad_table(gt, ref_gt)
