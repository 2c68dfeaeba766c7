"""GPU parity of the activation layer + lookup (Sec. 2.3) against the oracle.

Bars:
  * torus coordinates q: bit-exact (both sides form (K_i / 2 pi) arg z_i in fp64
    and round once to fp32); scale s: relative 1e-6 (fp64 on both sides,
    rounded to fp32 here);
  * theta forward per output row: relative L2 <= 1e-5 (fp32 table) or 2e-2
    (bf16 table, one rounding of the output);
  * grad_z and value-gradient rows (fp32 outputs): relative L2 <= 1e-5; rows
    no lookup touches stay exactly 0;
  * a zero or non-finite z_i: output and grad_z exactly 0.
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
    a = np.asarray(a, np.float64).reshape(a.shape[0], -1)
    b = np.asarray(b, np.float64).reshape(b.shape[0], -1)
    num = np.linalg.norm(a - b, axis=1)
    den = np.linalg.norm(b, axis=1)
    return np.where(den > 0, num / np.where(den > 0, den, 1), num)


def _z(L, seed, special=True):
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((L, 16)) * rng.uniform(0.05, 20.0, (L, 1))).astype(np.float32)
    if special:
        z[0] = 0
        z[0, 0::2] = 1.0                      # arg 0 everywhere: q = 0, a lattice point
        z[1] = 0
        z[1, 1::2] = 1.0                      # arg pi/2
        z[2] = 0
        z[2, 0::2] = -3.0                     # arg pi
        z[3, 6:8] = 0.0                       # z_3 = 0: scale 0
        z[4, 5] = np.inf
        z[5, 0] = np.nan
        z[6, 0::2] = np.abs(z[6, 0::2])       # right half-plane
        z[7, 1] = -0.0                        # signed zero imaginary part
    return z


def _table(K, m, dtype, seed=0):
    N = int(np.prod(K))
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn((N, m), generator=g, device=DEV) * 0.02).to(dtype)


@pytest.mark.parametrize("K", [(4,) * 8, (2, 4, 6, 8, 2, 4, 6, 8), (12,) * 8, (14,) * 8])
def test_theta_coords(K):
    _say("theta coords", K)
    z_np = _z(5000, 21)
    q, s = lram.theta_coords(torch.from_numpy(z_np).to(DEV), K)
    torch.cuda.synchronize()
    qr, sr = oracle.theta_coords(z_np, K)
    qg = q.cpu().numpy()
    fin = np.all(np.isfinite(z_np), axis=1)
    np.testing.assert_array_equal(qg[fin].view(np.uint32), qr[fin].view(np.uint32))
    assert np.all(np.isnan(qg[~fin, 0]))
    sg = s.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(sg, sr, rtol=1e-6, atol=0)


@pytest.mark.parametrize("mode", ["atomic", "merged", "sorted"])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("m", [32, 64])
@pytest.mark.parametrize("K", [(4,) * 8, (2, 4, 6, 8, 2, 4, 6, 8)])
def test_theta_forward_backward(K, m, dtype, mode):
    _say("theta fwd/bwd", K, m, dtype, mode)
    L = 3001
    z_np = _z(L, 22)
    z = torch.from_numpy(z_np).to(DEV)
    table = _table(K, m, dtype)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(100 + m + 7 * K[0] + (dtype == torch.bfloat16))
    G = torch.randn((L, m), device=DEV, generator=gen)
    out = lram.theta_forward(z, table, K)
    gt, gz = lram.theta_backward(z, table, K, G, mode=mode)
    qg, _ = lram.theta_coords(z, K)
    torch.cuda.synchronize()
    q, s = oracle.theta_coords(z_np, K)
    fin = np.all(np.isfinite(z_np), axis=1)
    np.testing.assert_array_equal(qg.cpu().numpy()[fin].view(np.uint32), q[fin].view(np.uint32))
    nb = oracle.neighbors(q, K)
    rows = oracle.gather_rows(table.float().cpu().numpy(), nb["slot"])
    ref = oracle.theta_forward(nb, rows, s)
    assert _rel_rows(out.float().cpu().numpy(), ref).max() <= (1e-5 if dtype == torch.float32 else 2e-2)
    Gn = G.cpu().numpy()
    gz_ref = oracle.theta_grad_z(z_np, K, nb, rows, s, Gn)
    err = _rel_rows(gz.cpu().numpy(), gz_ref)
    if err.max() > 1e-5:
        i = int(np.argmax(err))
        dq64 = oracle.grad_query(nb, rows, Gn)[i]
        dls64 = float(Gn[i] @ oracle.forward(nb, rows)[i])
        _say("worst row", i, "err", err[i], "s", s[i], "|z_i|", np.hypot(z_np[i, 0::2], z_np[i, 1::2]),
             "dq", dq64, "dL/ds", dls64, "count", nb["count"][i], "d2 max", nb["d2"][i].max(),
             "gpu", gz.cpu().numpy()[i], "ref", gz_ref[i])
    assert err.max() <= 1e-5, err.max()
    uniq, acc = oracle.theta_grad_table_rows(nb, s, Gn)
    dV = gt.cpu().numpy()
    live = np.abs(acc).max(axis=1) > 0          # rows reached only by scale-0 lookups stay 0
    assert _rel_rows(dV[uniq[live]], acc[live]).max() <= 1e-5
    mask = np.ones(dV.shape[0], bool)
    mask[uniq[live]] = False
    assert np.all(dV[mask] == 0)
    dead = np.array([3, 4, 5])
    assert np.all(out.float().cpu().numpy()[dead] == 0) and np.all(gz.cpu().numpy()[dead] == 0)


def test_theta_homogeneous_and_autograd():
    """theta(4 z) = 4 theta(z) on the GPU too (powers of two scale exactly), and
    the autograd wrapper returns the ABI's gradients."""
    K = (8,) * 8
    z = torch.from_numpy(_z(2000, 23, special=False)).to(DEV)
    table = _table(K, 32, torch.float32)
    o1 = lram.theta_forward(z, table, K)
    o4 = lram.theta_forward(z * 4, table, K)
    torch.cuda.synchronize()
    assert torch.equal(o4, 4 * o1)
    zr = z.clone().requires_grad_(True)
    tr = table.clone().requires_grad_(True)
    G = torch.randn((2000, 32), device=DEV)
    (lram.theta(zr, tr, K) * G).sum().backward()
    gt, gz = lram.theta_backward(z, table, K, G)
    torch.cuda.synchronize()
    assert torch.equal(zr.grad, gz)
    np.testing.assert_allclose(tr.grad.cpu().numpy(), gt.cpu().numpy(), rtol=1e-5, atol=1e-7)


@pytest.mark.parametrize("name", ["k4-m32-f32-gmm64", "k12-m64-bf16-proj"])
def test_theta_workload(name):
    """The workload's queries reached through the activation layer."""
    w = W.WORKLOADS[name]
    _say("theta workload", name)
    z_np = W.theta_inputs(w)
    z = torch.from_numpy(z_np).to(DEV)
    table = W.make_table(w, DEV)
    G = W.grad_out(w, DEV)
    out = lram.theta_forward(z, table, w.K)
    gt, gz = lram.theta_backward(z, table, w.K, G)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    zf = z_np.reshape(-1, 16)
    idx = np.sort(rng.choice(zf.shape[0], min(4096, zf.shape[0]), replace=False))
    q, s = oracle.theta_coords(zf[idx], w.K)
    nb = oracle.neighbors(q, w.K)
    ti = torch.from_numpy(np.maximum(nb["slot"], 0).astype(np.int64)).to(DEV)
    rows = table[ti].float().cpu().numpy().astype(np.float64)
    rows[nb["slot"] < 0] = 0
    ref = oracle.theta_forward(nb, rows, s)
    got = out.reshape(-1, w.m)[torch.from_numpy(idx).to(DEV)].float().cpu().numpy()
    assert _rel_rows(got, ref).max() <= (1e-5 if w.dtype == "f32" else 2e-2)
    Gs = G.reshape(-1, w.m)[torch.from_numpy(idx).to(DEV)].cpu().numpy()
    gz_ref = oracle.theta_grad_z(zf[idx], w.K, nb, rows, s, Gs)
    assert _rel_rows(gz.reshape(-1, 16)[torch.from_numpy(idx).to(DEV)].cpu().numpy(), gz_ref).max() <= 1e-5
