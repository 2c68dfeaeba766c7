"""Reference oracle for the LRAM lattice lookup -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The product library never imports, links or calls it, and it
never imports the product: the two share nothing but the seeded input
generators in ``workloads.py``.

What it computes (Goucher & Troll, "Differentiable Random Access Memory using
Lattices"):

* ``neighbors``  -- the closest 32 lattice points of Lambda = 2*E8 (Sec. 2.4)
  within the kernel support r^2 < 8 (Sec. 2.5, Sec. 2.6), enumerated straight
  from the definition by the C helper ``lram_oracle.c``; their locations on the
  torus (Sec. 2.2), the fp32 recipe distances that decide the selection and
  the kernel weights f(r) = (1 - r^2/8)^4 in fp64.  ``k`` = 16 or 64 keeps
  that many instead, ``k`` = 0 every point of the support (the untruncated
  sum of Sec. 2.2 / 2.5).
* ``forward``    -- phi_32(q) = sum_j w_j v_{slot_j} (Sec. 2.2 with the
  truncation of Sec. 2.6), accumulated in fp64.
* ``backward``   -- the gradients of <G, phi_32(q)> with respect to the value
  table (dV[s] = sum over (l,j) with slot_j(l) = s of w_j G_l) and to the query
  (dq_i = sum_j -2 u_j^3 (x_i - k_{j,i}) <G, v_j>, u = 1 - r^2/8, the factor 2
  being dx/dq), with the selection held fixed (Sec. 2.6: the kernel returns
  the weights and their partial derivatives for an autograd wrapper).

* ``theta_*``    -- the activation layer of Sec. 2.3 in front of the lookup:
  theta(z) = (sum_i 1/|z_i|)^-1 phi_32((K_i / 2 pi) arg z_i) for z in C^8,
  given as 16 reals (Re z_0, Im z_0, ..., Re z_7, Im z_7), and its gradients
  with respect to z (through arg and the scale) and to the value table.
* ``sparse_adam`` -- one Adam step (Sec. 3.2 trains the memory with Adam at
  learning rate 1e-3) applied only to the rows whose gradient is not all zero.
* ``access_histogram``, ``access_stats`` -- the weighted access count of every
  location and, from it, the share of locations used and the KL divergence
  of the access distribution from uniform (the statistics of Sec. 4.3).
* ``oracle.subnetwork`` -- the memory subnetwork of Sec. 3.1 around theta.

Scale and the other readings of the paper are stated in the header of
``lram_oracle.c``.  All functions take numpy arrays on the host.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

NB = 32
_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lram_oracle.c")
_BUILD = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD, "liblram_oracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the C helper with gcc (OpenMP, no FP contraction)."""
    os.makedirs(_BUILD, exist_ok=True)
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-ffp-contract=off", "-fno-fast-math", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_LIB_PATH)
            P = ctypes.c_void_p
            lib.lram_oracle_neighbors.argtypes = [P, ctypes.c_int64, P, P, P, P, P, P, P, P, P, P]
            lib.lram_oracle_neighbors.restype = ctypes.c_int
            lib.lram_oracle_neighbors_k.argtypes = [P, ctypes.c_int64, P, ctypes.c_int32, P, P, P, P, P, P, P, P, P]
            lib.lram_oracle_neighbors_k.restype = ctypes.c_int
            lib.lram_oracle_locations.argtypes = [P, ctypes.c_int64, P, P]
            lib.lram_oracle_locations.restype = None
            lib.lram_oracle_recipe_d2.argtypes = [P, P, ctypes.c_int64, P]
            lib.lram_oracle_recipe_d2.restype = None
            _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check_k(K) -> np.ndarray:
    K = np.ascontiguousarray(np.asarray(K, dtype=np.int32).reshape(8))
    if np.any(K < 2) or np.any(K % 2):
        raise ValueError("every K_i must be even and >= 2")
    if np.prod(K.astype(np.int64)) >= 2 ** 31:
        raise ValueError("N = prod(K) must be below 2^31 (int32 locations)")
    return K


ALL_WIDTH = 256  # list width of the untruncated lookup (the support holds at most 241 points)


def neighbors(q: np.ndarray, K, k: int = 32) -> dict:
    """Closest-k neighbour lists of queries q[..., 8] (user scale) on torus K.

    k = 32 is the truncation of Sec. 2.6; other k keep the closest min(k, count)
    points in the same order; k = 0 keeps the whole support (the untruncated
    sum of Sec. 2.2 / 2.5) in lists of width ALL_WIDTH."""
    K = _check_k(K)
    width = ALL_WIDTH if k == 0 else int(k)
    if width < 1:
        raise ValueError("k must be positive, or 0 for the whole support")
    q = np.ascontiguousarray(np.asarray(q, dtype=np.float32))
    lead = q.shape[:-1]
    assert q.shape[-1] == 8
    qf = q.reshape(-1, 8)
    L = qf.shape[0]
    x = np.empty((L, 8), np.float32)
    count = np.empty(L, np.int32)
    slot = np.empty((L, width), np.int32)
    d2 = np.empty((L, width), np.float32)
    d64 = np.empty((L, width), np.float64)
    w64 = np.empty((L, width), np.float64)
    w32 = np.empty((L, width), np.float32)
    lift = np.empty((L, width, 8), np.int32)
    wsum = np.empty(L, np.float64)
    if L:
        rc = _load().lram_oracle_neighbors_k(_ptr(qf), L, _ptr(K), ctypes.c_int32(width), _ptr(x), _ptr(count),
                                             _ptr(slot), _ptr(d2), _ptr(d64), _ptr(w64), _ptr(w32), _ptr(lift),
                                             _ptr(wsum))
        if rc != 0:
            raise RuntimeError("oracle: support larger than expected")
    out = dict(x=x, count=count, slot=slot, d2=d2, d64=d64, w64=w64, w32=w32, lift=lift, wsum=wsum)
    return {k: v.reshape(lead + v.shape[1:]) for k, v in out.items()}


def locations(k: np.ndarray, K) -> np.ndarray:
    """Location index of explicit lattice points k[..., 8] (Lambda scale)."""
    K = _check_k(K)
    k = np.ascontiguousarray(np.asarray(k, dtype=np.int32))
    lead = k.shape[:-1]
    kf = k.reshape(-1, 8)
    out = np.empty(kf.shape[0], np.int32)
    if kf.shape[0]:
        _load().lram_oracle_locations(_ptr(kf), kf.shape[0], _ptr(K), _ptr(out))
    return out.reshape(lead)


def recipe_d2(x: np.ndarray, k: np.ndarray) -> np.ndarray:
    """The fp32 distance recipe for explicit pairs x[...,8] (fp32), k[...,8] (int)."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    k = np.ascontiguousarray(np.broadcast_to(np.asarray(k, dtype=np.int32), x.shape))
    lead = x.shape[:-1]
    out = np.empty(int(np.prod(lead)) if lead else 1, np.float32)
    if out.size:
        _load().lram_oracle_recipe_d2(_ptr(x.reshape(-1, 8)), _ptr(k.reshape(-1, 8)), out.size, _ptr(out))
    return out.reshape(lead)


def gather_rows(table: np.ndarray, slot: np.ndarray) -> np.ndarray:
    """rows[..., j, :] = table[slot[..., j]] in fp64 (zero rows for slot -1)."""
    t = np.asarray(table, dtype=np.float64)
    s = np.asarray(slot)
    rows = t[np.where(s >= 0, s, 0)]
    rows[s < 0] = 0.0
    return rows


def forward(nb: dict, rows: np.ndarray) -> np.ndarray:
    """phi_32 = sum_j w_j v_{slot_j}, fp64; rows[..., 32, m] are the value rows."""
    w = nb["w64"]
    return np.einsum("...j,...jm->...m", w, np.asarray(rows, np.float64))


def grad_query(nb: dict, rows: np.ndarray, G: np.ndarray) -> np.ndarray:
    """dq[..., i] = sum_j -2 u_j^3 (x_i - k_{j,i}) <G, v_j>  (user-scale q), fp64."""
    G = np.asarray(G, np.float64)
    gv = np.einsum("...m,...jm->...j", G, np.asarray(rows, np.float64))
    u = 1.0 - nb["d64"] / 8.0
    valid = nb["slot"] >= 0
    a = np.where(valid, -2.0 * u ** 3 * gv, 0.0)
    e = nb["x"].astype(np.float64)[..., None, :] - nb["lift"].astype(np.float64)
    # padded entries (and every entry of a non-finite query) contribute nothing
    e = np.where(valid[..., None], e, 0.0)
    return np.einsum("...j,...ji->...i", a, e)


def grad_table_rows(nb: dict, G: np.ndarray, weights: str = "w64"):
    """Value-table gradient as (unique slots, rows): dV[s] = sum_{(l,j): slot=s} w_j G_l, fp64.

    ``weights`` picks the kernel weights: "w64" (fp64 distance, the default)
    or "w32" (the fp32 recipe weights, for comparisons in which the weights of
    neighbours at the edge of the support, u = 1 - r^2/8 near the fp32
    resolution of r^2, must not dominate a row)."""
    G = np.asarray(G, np.float64)
    m = G.shape[-1]
    width = nb["slot"].shape[-1]
    slot = nb["slot"].reshape(-1, width)
    w = nb[weights].reshape(-1, width).astype(np.float64)
    Gf = G.reshape(-1, m)
    valid = slot >= 0
    s = slot[valid]
    contrib = (w[:, :, None] * Gf[:, None, :])[valid]
    uniq, inv = np.unique(s, return_inverse=True)
    acc = np.zeros((uniq.size, m), np.float64)
    np.add.at(acc, inv, contrib)
    return uniq.astype(np.int64), acc


def grad_table_dense(nb: dict, G: np.ndarray, N: int) -> np.ndarray:
    uniq, acc = grad_table_rows(nb, G)
    out = np.zeros((N, acc.shape[1] if acc.ndim == 2 else np.asarray(G).shape[-1]), np.float64)
    out[uniq] = acc
    return out


# ---------------------------------------------------------------------------
# Activation layer (Sec. 2.3).

def theta_coords(z: np.ndarray, K):
    """Torus coordinates and output scale of theta for z[..., 16] (Sec. 2.3).

    q_i = (K_i / (2 pi)) * arg z_i, formed in fp64 and rounded once to fp32
    (the query precision of the lookup); s = (sum_i 1/|z_i|)^-1 in fp64 -- the
    displayed formula of Sec. 2.3, which the text calls a harmonic mean
    (without its factor n).  A zero z_i gives s = 0 (the continuous
    extension); a non-finite input gives a NaN query (empty neighbour list)
    and s = 0.
    """
    K = _check_k(K)
    z = np.asarray(np.asarray(z, np.float32), np.float64)
    assert z.shape[-1] == 16
    a, b = z[..., 0::2], z[..., 1::2]
    c = K.astype(np.float64) / (2.0 * np.pi)
    finite = np.all(np.isfinite(z), axis=-1)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        q = (np.arctan2(b, a) * c).astype(np.float32)
        s = 1.0 / np.sum(1.0 / np.hypot(a, b), axis=-1)
    q = np.where(finite[..., None], q, np.float32(np.nan))
    s = np.where(finite, s, 0.0)
    return q, s


def theta_forward(nb: dict, rows: np.ndarray, s: np.ndarray) -> np.ndarray:
    """theta = s * phi_32(q), fp64 (nb and rows of the queries from theta_coords)."""
    return np.asarray(s, np.float64)[..., None] * forward(nb, rows)


def theta_grad_table_rows(nb: dict, s: np.ndarray, G: np.ndarray, weights: str = "w64"):
    """Value-table gradient of <G, theta>: the lookup's with G scaled by s."""
    return grad_table_rows(nb, np.asarray(G, np.float64) * np.asarray(s, np.float64)[..., None], weights)


def theta_grad_z(z: np.ndarray, K, nb: dict, rows: np.ndarray, s: np.ndarray, G: np.ndarray) -> np.ndarray:
    """d<G, theta>/dz[..., 16] (selection held fixed), fp64.

    With r_i = |z_i|, t_i = arg z_i, q_i = c_i t_i, c_i = K_i / (2 pi):
    ds/da_i = s^2 a_i / r_i^3, ds/db_i = s^2 b_i / r_i^3 (from s = 1 / sum 1/r),
    dt_i/da_i = -b_i / r_i^2, dt_i/db_i = a_i / r_i^2, and
    d<G, theta>/ds = <G, phi>, d<G, theta>/dq = s * (dq of the lookup for G).
    Zero where s = 0 (a zero or non-finite entry).
    """
    K = _check_k(K)
    z = np.asarray(np.asarray(z, np.float32), np.float64)
    a, b = z[..., 0::2], z[..., 1::2]
    c = K.astype(np.float64) / (2.0 * np.pi)
    s = np.asarray(s, np.float64)
    G = np.asarray(G, np.float64)
    dLds = np.einsum("...m,...m->...", G, forward(nb, rows))
    dLdq = s[..., None] * grad_query(nb, rows, G)
    ok = s > 0
    with np.errstate(divide="ignore", invalid="ignore"):
        r2 = a * a + b * b
        r3 = r2 * np.sqrt(r2)
        ga = dLds[..., None] * s[..., None] ** 2 * a / r3 - dLdq * c * b / r2
        gb = dLds[..., None] * s[..., None] ** 2 * b / r3 + dLdq * c * a / r2
    out = np.empty(z.shape, np.float64)
    out[..., 0::2] = np.where(ok[..., None], ga, 0.0)
    out[..., 1::2] = np.where(ok[..., None], gb, 0.0)
    return out


# ---------------------------------------------------------------------------
# Training-side companions: the optimiser step on the memory table (Sec. 3.2:
# Adam, learning rate 1e-3 for the memory parameters) and the access
# statistics of Sec. 4.3 (Table 5).

def sparse_adam(table, grad, exp_avg, exp_avg_sq, step, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8):
    """One Adam step (Kingma & Ba, Algorithm 1: bias-corrected moments, eps
    outside the square root) on the rows of the table whose gradient row is not
    identically zero; the other rows keep their values and moments (the lazy,
    sparse form).  fp64; returns new (table, exp_avg, exp_avg_sq)."""
    V = np.array(table, np.float64)
    g = np.asarray(grad, np.float64)
    m1 = np.array(exp_avg, np.float64)
    m2 = np.array(exp_avg_sq, np.float64)
    rows = np.any(g != 0, axis=1)
    m1[rows] = beta1 * m1[rows] + (1 - beta1) * g[rows]
    m2[rows] = beta2 * m2[rows] + (1 - beta2) * g[rows] ** 2
    mh = m1[rows] / (1 - beta1 ** step)
    vh = m2[rows] / (1 - beta2 ** step)
    V[rows] = V[rows] - lr * mh / (np.sqrt(vh) + eps)
    return V, m1, m2


def access_histogram(nb: dict, N: int, weights: str = "w64") -> np.ndarray:
    """Weighted access count of every location: sum of the kernel weights of
    the (lookup, neighbour) pairs that read it (fp64; ``weights`` as in
    grad_table_rows)."""
    s = nb["slot"].reshape(-1)
    w = nb[weights].reshape(-1).astype(np.float64)
    ok = s >= 0
    return np.bincount(s[ok], weights=w[ok], minlength=N).astype(np.float64)


def access_stats(hist: np.ndarray):
    """(fraction of locations accessed, KL divergence of the weighted access
    distribution from uniform) -- the two columns of Table 5."""
    h = np.asarray(hist, np.float64)
    N = h.size
    tot = h.sum()
    p = h[h > 0] / tot
    return float((h > 0).mean()), float(np.sum(p * np.log(p * N)))
