"""GPU parity of the memory subnetwork (Sec. 3.1): dense w -> w, batch norm of
the queries, theta (n, m, h) = (8, 64, w/16) through liblram, dense 4w -> w,
against the fp64 oracle of the same slice.

The input layer is made exact (dyadic inputs and weights whose fp32 products
and sums round nowhere; inference-form normalisation with unit variance),
so the queries, and with them the neighbour selection, are the
oracle's bit for bit (torch requires eps > 0: eps = 2^-20 with running
variance 1 - 2^-20 sums to 1 exactly); the rest is compared at the fp32 bar: per-row relative
L2 <= 1e-5 for y and every gradient (value-table rows against the fp64 sum of
the recipe weights, whose lists are pinned bit-exactly elsewhere).

Training form (batch statistics; Sec. 4.1 normalises the queries while
training): torch forms the batch mean and variance in fp32, which no fp64
evaluation reproduces bit for bit, so the normalised queries are compared
with the oracle's training-form normalisation at 1e-5 and the oracle's lookup
then takes the same fp32 queries (its neighbour selection is compared bit for
bit elsewhere); y and every gradient, through the batch statistics, at 1e-5;
the b1 gradient, zero in exact arithmetic, within 1e-5 of the beta gradient's
size.
"""
import numpy as np
import pytest
import torch

from oracle import subnetwork as sub
from paper_2107_03474_amd.memory_layer import MemorySubnetwork

pytestmark = pytest.mark.gpu
DEV = "cuda"
K = (4, 6, 4, 6, 4, 6, 4, 6)


def _rel_rows(a, b):
    a = np.asarray(a, np.float64).reshape(a.shape[0], -1)
    b = np.asarray(b, np.float64).reshape(b.shape[0], -1)
    num = np.linalg.norm(a - b, axis=1)
    den = np.linalg.norm(b, axis=1)
    return np.where(den > 0, num / np.where(den > 0, den, 1), num)


@pytest.mark.parametrize("scatter", ["atomic", "merged"])
def test_subnetwork_parity(scatter):
    w, T = 512, 256
    rng = np.random.default_rng(41)
    torch.manual_seed(41)
    net = MemorySubnetwork(w, K, table_dtype=torch.float32, device=DEV, scatter=scatter).eval()
    x = (rng.integers(-1, 2, (T, w)) / 4.0).astype(np.float32)
    W1 = (rng.integers(-3, 4, (w, w)) / 64.0).astype(np.float32)
    b1 = (rng.integers(-3, 4, w) / 64.0).astype(np.float32)
    mu = (rng.integers(-2, 3, w) / 16.0).astype(np.float32)
    gamma = (2.0 ** rng.integers(-1, 2, w)).astype(np.float32)
    beta = (rng.integers(-2, 3, w) / 16.0).astype(np.float32)
    with torch.no_grad():
        net.inp.weight.copy_(torch.from_numpy(W1))
        net.inp.bias.copy_(torch.from_numpy(b1))
        net.bn.running_mean.copy_(torch.from_numpy(mu))
        net.bn.running_var.fill_(1.0 - 2.0 ** -20)   # var + eps = 1 exactly in fp32
        net.bn.eps = 2.0 ** -20
        net.bn.weight.copy_(torch.from_numpy(gamma))
        net.bn.bias.copy_(torch.from_numpy(beta))
    xt = torch.from_numpy(x).to(DEV).requires_grad_(True)
    y = net(xt)
    dy = torch.randn_like(y)
    y.backward(dy)
    torch.cuda.synchronize()

    p = {"W1": W1.astype(np.float64), "b1": b1.astype(np.float64), "mu": mu.astype(np.float64),
         "var": np.full(w, 1.0 - 2.0 ** -20), "eps": 2.0 ** -20, "gamma": gamma.astype(np.float64),
         "beta": beta.astype(np.float64),
         "W2": net.out.weight.detach().cpu().numpy().astype(np.float64),
         "b2": net.out.bias.detach().cpu().numpy().astype(np.float64)}
    table = net.table.detach().cpu().numpy().astype(np.float64)
    y_ref, st = sub.forward(x, p, K, table)
    # the exact input layer gives the oracle's queries bit for bit
    z_gpu = net.bn(net.inp(torch.from_numpy(x).to(DEV))).detach().cpu().numpy()
    np.testing.assert_array_equal(z_gpu.reshape(st["z"].shape), st["z"].astype(np.float32))
    assert _rel_rows(y.detach().cpu().numpy(), y_ref).max() <= 1e-5
    g = sub.backward(dy.cpu().numpy(), p, K, table, st, table_weights="w32")
    checks = {"x": xt.grad, "W1": net.inp.weight.grad, "b1": net.inp.bias.grad[None], "gamma": net.bn.weight.grad[None],
              "beta": net.bn.bias.grad[None], "W2": net.out.weight.grad, "b2": net.out.bias.grad[None]}
    for name, got in checks.items():
        ref = g[name] if g[name].ndim == 2 else g[name][None]
        err = _rel_rows(got.cpu().numpy(), ref)
        assert err.max() <= 1e-5, (name, err.max())
    uniq, acc = g["table"]
    gt = net.table.grad.cpu().numpy()
    assert _rel_rows(gt[uniq], acc).max() <= 1e-5
    mask = np.ones(gt.shape[0], bool)
    mask[uniq] = False
    assert np.all(gt[mask] == 0)


@pytest.mark.parametrize("scatter", ["atomic", "merged"])
def test_subnetwork_parity_training(scatter):
    w, T = 512, 256
    rng = np.random.default_rng(43)
    torch.manual_seed(43)
    net = MemorySubnetwork(w, K, table_dtype=torch.float32, device=DEV, scatter=scatter).train()
    x = rng.standard_normal((T, w)).astype(np.float32)
    with torch.no_grad():
        net.bn.weight.copy_(torch.from_numpy(rng.uniform(0.5, 1.5, w).astype(np.float32)))
        net.bn.bias.copy_(torch.from_numpy((rng.standard_normal(w) * 0.1).astype(np.float32)))
    xt = torch.from_numpy(x).to(DEV).requires_grad_(True)
    y = net(xt)
    with torch.no_grad():
        z_gpu = net.bn(net.inp(torch.from_numpy(x).to(DEV))).cpu().numpy()
    dy = torch.randn_like(y)
    y.backward(dy)
    torch.cuda.synchronize()
    f64 = lambda t: t.detach().cpu().numpy().astype(np.float64)
    p = {"W1": f64(net.inp.weight), "b1": f64(net.inp.bias), "mu": np.zeros(w), "var": np.ones(w),
         "eps": float(net.bn.eps), "gamma": f64(net.bn.weight), "beta": f64(net.bn.bias),
         "W2": f64(net.out.weight), "b2": f64(net.out.bias)}
    table = f64(net.table)
    y_ref, st = sub.forward(x, p, K, table, training=True, queries=z_gpu)
    assert _rel_rows(z_gpu, st["z"].reshape(T, w)).max() <= 1e-5
    assert _rel_rows(y.detach().cpu().numpy(), y_ref).max() <= 1e-5
    g = sub.backward(dy.cpu().numpy(), p, K, table, st, table_weights="w32")
    checks = {"x": xt.grad, "W1": net.inp.weight.grad, "gamma": net.bn.weight.grad[None],
              "beta": net.bn.bias.grad[None], "W2": net.out.weight.grad, "b2": net.out.bias.grad[None]}
    for name, got in checks.items():
        ref = g[name] if g[name].ndim == 2 else g[name][None]
        err = _rel_rows(got.cpu().numpy(), ref)
        assert err.max() <= 1e-5, (name, err.max())
    gb1 = net.inp.bias.grad.cpu().numpy()
    assert np.linalg.norm(gb1) <= 1e-5 * np.linalg.norm(g["beta"])
    uniq, acc = g["table"]
    gt = net.table.grad.cpu().numpy()
    assert _rel_rows(gt[uniq], acc).max() <= 1e-5
    mask = np.ones(gt.shape[0], bool)
    mask[uniq] = False
    assert np.all(gt[mask] == 0)
