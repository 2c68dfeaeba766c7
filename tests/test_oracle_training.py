"""Pins of the oracle's optimiser step and access statistics.

* Adam: on a table whose every row is touched the step is torch's own
  ``torch.optim.Adam`` (a library routine, CPU fp64), repeated over several
  steps; untouched rows keep values and moments exactly; the first step moves
  each touched entry by lr * g / (|g| + eps) against its gradient.
* Access statistics: queries at every lattice point of a small torus read
  each location once with weight 1 (used = 1, KL = 0); repeating the batch
  changes neither statistic; a single lookup's KL is log N minus the entropy
  of its normalised weights.
"""
import itertools

import numpy as np
import torch

import oracle


def test_adam_matches_torch_when_every_row_is_touched():
    rng = np.random.default_rng(1)
    N, m = 50, 8
    V0 = rng.standard_normal((N, m))
    p = torch.nn.Parameter(torch.from_numpy(V0.copy()))
    opt = torch.optim.Adam([p], lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    V, m1, m2 = V0.copy(), np.zeros((N, m)), np.zeros((N, m))
    for t in range(1, 6):
        g = rng.standard_normal((N, m))
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        V, m1, m2 = oracle.sparse_adam(V, g, m1, m2, t)
        np.testing.assert_allclose(V, p.detach().numpy(), rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(m1, opt.state[p]["exp_avg"].numpy(), rtol=1e-12)  # torch uses lerp
        np.testing.assert_allclose(m2, opt.state[p]["exp_avg_sq"].numpy(), rtol=1e-12)


def test_adam_is_lazy_on_untouched_rows_and_first_step_closed_form():
    rng = np.random.default_rng(2)
    N, m = 40, 4
    V0 = rng.standard_normal((N, m))
    g = rng.standard_normal((N, m))
    g[::3] = 0.0
    m1 = rng.standard_normal((N, m)) * 0.1
    m2 = rng.random((N, m)) * 0.1
    V, n1, n2 = oracle.sparse_adam(V0, g, m1, m2, 7)
    assert np.all(V[::3] == V0[::3]) and np.all(n1[::3] == m1[::3]) and np.all(n2[::3] == m2[::3])
    V1, _, _ = oracle.sparse_adam(V0, g, np.zeros((N, m)), np.zeros((N, m)), 1, lr=1e-3, eps=1e-8)
    touched = np.any(g != 0, axis=1)
    np.testing.assert_allclose(V1[touched], V0[touched] - 1e-3 * g[touched] / (np.abs(g[touched]) + 1e-8),
                               rtol=1e-12)


def _all_points(K):
    """Every lattice point of the torus K (coset representatives at the Lambda
    scale, as user-scale queries q = k / 2)."""
    pts = []
    for eps in (0, 1):
        for Y in itertools.product(*[range(k) for k in K]):
            if sum(Y) % 2 == 0:
                pts.append((2 * np.asarray(Y) + eps) / 2.0)
    return np.asarray(pts, np.float32)


def test_stats_uniform_at_lattice_points():
    K = (2, 2, 2, 4, 2, 2, 2, 2)
    N = int(np.prod(K))
    q = _all_points(K)
    assert q.shape[0] == N
    nb = oracle.neighbors(q, K)
    h = oracle.access_histogram(nb, N)
    np.testing.assert_allclose(h, 1.0, rtol=1e-15)
    used, kl = oracle.access_stats(h)
    assert used == 1.0 and abs(kl) < 1e-12


def test_stats_scale_invariance_and_single_lookup():
    K = (4,) * 8
    N = 4 ** 8
    rng = np.random.default_rng(3)
    q = (rng.random((300, 8)) * 4).astype(np.float32)
    nb = oracle.neighbors(q, K)
    h = oracle.access_histogram(nb, N)
    nb2 = oracle.neighbors(np.concatenate([q, q]), K)
    h2 = oracle.access_histogram(nb2, N)
    assert oracle.access_stats(h) == (oracle.access_stats(h2)[0], oracle.access_stats(h)[1])
    np.testing.assert_allclose(oracle.access_stats(h2)[1], oracle.access_stats(h)[1], rtol=1e-12)
    one = oracle.neighbors(q[:1], K)
    w = one["w64"][0][one["slot"][0] >= 0]
    pw = w / w.sum()
    used, kl = oracle.access_stats(oracle.access_histogram(one, N))
    assert used == w.size / N
    np.testing.assert_allclose(kl, np.log(N) + np.sum(pw * np.log(pw)), rtol=1e-12)
