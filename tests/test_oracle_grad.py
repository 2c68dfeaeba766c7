"""Gradients of the oracle: central finite differences for dq, the adjoint identity for dV.

The query gradient is the derivative of <G, phi_32(q)> with the truncated
selection held fixed (Sec. 2.6: the kernel reports the weights and their partial
derivatives for an autograd wrapper); queries where the selection changes within
the step are skipped.
"""
import numpy as np
import pytest

import oracle


@pytest.mark.parametrize("K", [(4,) * 8, (8,) * 8, (2,) * 8])
def test_dq_matches_central_differences(K):
    rng = np.random.default_rng(21)
    N = int(np.prod(K))
    m = 8
    table = rng.standard_normal((N, m))
    # dyadic queries so that q +- h is exact in fp32 and x = 2q stays exact
    q = (rng.integers(0, 2 ** 12 * K[0], size=(40, 8)) / 2 ** 12).astype(np.float32)
    G = rng.standard_normal((40, m))
    h = 2.0 ** -14
    nb = oracle.neighbors(q, K)
    rows = oracle.gather_rows(table, nb["slot"])
    dq = oracle.grad_query(nb, rows, G)
    checked = 0
    for l in range(q.shape[0]):
        for i in range(8):
            qp = q[l:l + 1].copy()
            qm = q[l:l + 1].copy()
            qp[0, i] += np.float32(h)
            qm[0, i] -= np.float32(h)
            assert qp[0, i] - q[l, i] == np.float32(h)
            nbp = oracle.neighbors(qp, K)
            nbm = oracle.neighbors(qm, K)
            if not (np.array_equal(nbp["slot"][0], nb["slot"][l]) and np.array_equal(nbm["slot"][0], nb["slot"][l])):
                continue
            fp = G[l] @ oracle.forward(nbp, oracle.gather_rows(table, nbp["slot"]))[0]
            fm = G[l] @ oracle.forward(nbm, oracle.gather_rows(table, nbm["slot"]))[0]
            fd = (fp - fm) / (2 * h)
            assert abs(fd - dq[l, i]) <= 1e-6 * (1 + abs(dq[l, i])), (l, i, fd, dq[l, i])
            checked += 1
    assert checked > 200


@pytest.mark.parametrize("K", [(4,) * 8, (2,) * 8, (2, 4, 2, 4, 4, 2, 4, 2)])
def test_table_gradient_adjoint(K):
    """<G, phi_{dV}(Q)> = <grad_V(G), dV>: phi is linear in the table (Sec. 2.2).
    At K = 2 one location appears through two lifts, so accumulation matters."""
    rng = np.random.default_rng(22)
    N = int(np.prod(K))
    m = 5
    q = (rng.random((300, 8)) * np.asarray(K)).astype(np.float32)
    G = rng.standard_normal((300, m))
    dV = rng.standard_normal((N, m))
    nb = oracle.neighbors(q, K)
    lhs = np.sum(G * oracle.forward(nb, oracle.gather_rows(dV, nb["slot"])))
    gV = oracle.grad_table_dense(nb, G, N)
    rhs = np.sum(gV * dV)
    assert abs(lhs - rhs) <= 1e-10 * (1 + abs(lhs))
    untouched = np.setdiff1d(np.arange(N), nb["slot"][nb["slot"] >= 0])
    assert np.all(gV[untouched] == 0)
