"""Seeded synthetic inputs for the LRAM lookup workloads.

Shared by the tests, the smoke check and the benchmark.  This module holds no
lattice arithmetic: it only draws random queries, value tables and upstream
gradients with the shapes and distributions of the named workloads.  The paper's
language-modelling data (Sec. 3.3) and trained weights are not available, so
these inputs stand in for them; they are not reproductions.

Random streams: numpy PCG64 children of SeedSequence(seed), spawned in a fixed
order (queries, mixture, projection); value tables and upstream gradients are
drawn on the target device with a seeded torch.Generator in fixed-size chunks.
"""
from __future__ import annotations

import dataclasses
from typing import Tuple

import numpy as np

TABLE_STD = 0.02


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    K: Tuple[int, ...]
    m: int
    dtype: str            # "f32" or "bf16" table
    B: int
    H: int
    queries: str          # "uniform", "gmm", "projection", "zipf_mix"
    backward: bool
    gmm_components: int = 0
    gmm_sigma: float = 0.0
    zipf_centres: int = 0
    zipf_s: float = 0.0
    proj_in: int = 0
    desc: str = ""

    @property
    def N(self) -> int:
        return int(np.prod(self.K))

    @property
    def L(self) -> int:
        return self.B * self.H

    @property
    def table_bytes(self) -> int:
        return self.N * self.m * (4 if self.dtype == "f32" else 2)


WORKLOADS = {
    "k4-m32-f32-uniform": Workload(
        "k4-m32-f32-uniform", (4,) * 8, 32, "f32", 4096, 1, "uniform", True,
        desc="K=(4,..,4), 65,536 locations, m=32 fp32 table ~N(0,0.02); 4,096 x 1 uniform queries; fwd+bwd"),
    "k8-m64-f32-uniform": Workload(
        "k8-m64-f32-uniform", (8,) * 8, 64, "f32", 65536, 8, "uniform", False,
        desc="K=(8,..,8), 16,777,216 locations, m=64 fp32 table (4.3 GB); 65,536 x 8 uniform queries; fwd"),
    "k4-m32-f32-gmm64": Workload(
        "k4-m32-f32-gmm64", (4,) * 8, 32, "f32", 4096, 1, "gmm", True, gmm_components=64, gmm_sigma=0.3,
        desc="the K=4 table; 4,096 x 1 queries from an equal-weight 64-component Gaussian mixture (sigma 0.3)"),
    "k12-m64-bf16-proj": Workload(
        "k12-m64-bf16-proj", (12,) * 8, 64, "bf16", 8192, 16, "projection", True, proj_in=1024,
        desc="BERT-style slice: 16x512 tokens, q = wrap(X W), X ~ N(0,1) [8192,1024], W ~ N(0,1/1024) "
             "[1024,128]; K=12, 429,981,696 locations, m=64 bf16 table (55 GB); fwd+bwd"),
    "k14-m32-bf16-zipf": Workload(
        "k14-m32-bf16-zipf", (14,) * 8, 32, "bf16", 262144, 16, "zipf_mix", True, gmm_sigma=0.3,
        zipf_centres=4096, zipf_s=1.1,
        desc="billion scale: K=14, 1,475,789,056 locations, m=32 bf16 table (94 GB) + fp32 gradient "
             "(189 GB); 262,144 x 16 queries, half uniform, half around 4,096 Zipf(1.1)-ranked centres"),
}


def _streams(seed: int):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(3)]


def _wrap(q: np.ndarray, K) -> np.ndarray:
    """Bring user-scale coordinates into [0, K_i) (plain floor-modulo); a value that
    rounds up to K_i in fp32 is the same torus point as 0 and is stored as 0."""
    Kf = np.asarray(K, np.float64)
    q32 = np.mod(q, Kf).astype(np.float32)
    return np.where(q32 >= Kf.astype(np.float32), np.float32(0), q32).astype(np.float32)


def queries(w: Workload, seed: int = 0) -> np.ndarray:
    """Queries [B, H, 8] fp32 (user scale, coordinates in [0, K_i))."""
    rq, rmix, rproj = _streams(seed)
    B = w.B
    Kf = np.asarray(w.K, np.float64)
    n = B * w.H
    if w.queries == "uniform":
        q = rq.random((n, 8)) * Kf
    elif w.queries == "gmm":
        mu = rmix.random((w.gmm_components, 8)) * Kf
        comp = rq.integers(0, w.gmm_components, size=n)
        q = mu[comp] + w.gmm_sigma * rq.standard_normal((n, 8))
    elif w.queries == "projection":
        W = rproj.standard_normal((w.proj_in, w.H * 8)) / np.sqrt(w.proj_in)
        X = rq.standard_normal((B, w.proj_in))
        q = (X @ W).reshape(n, 8)
    elif w.queries == "zipf_mix":
        mu = rmix.random((w.zipf_centres, 8)) * Kf
        p = np.arange(1, w.zipf_centres + 1, dtype=np.float64) ** (-w.zipf_s)
        p /= p.sum()
        clustered = np.zeros(n, bool)
        clustered[: n // 2] = True
        clustered = clustered[rmix.permutation(n)]
        comp = rmix.choice(w.zipf_centres, size=n, p=p)
        u = rq.random((n, 8)) * Kf
        g = mu[comp] + w.gmm_sigma * rq.standard_normal((n, 8))
        q = np.where(clustered[:, None], g, u)
    else:
        raise ValueError(w.queries)
    return _wrap(q, w.K).reshape(B, w.H, 8)


def theta_inputs(w: Workload, seed: int = 0) -> np.ndarray:
    """Inputs [B, H, 16] fp32 for the activation layer that land on the
    workload's queries: z_i = r_i (cos t_i, sin t_i) with t_i = 2 pi q_i / K_i
    (interleaved Re, Im) and moduli r_i ~ Rayleigh(1) (|N(0,1) + i N(0,1)| / sqrt 2,
    the modulus of a random complex projection)."""
    q = queries(w, seed).astype(np.float64)
    r = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed + 7))).rayleigh(1.0, q.shape)
    t = 2.0 * np.pi * q / np.asarray(w.K, np.float64)
    z = np.empty(q.shape[:-1] + (16,), np.float32)
    z[..., 0::2] = r * np.cos(t)
    z[..., 1::2] = r * np.sin(t)
    return z


def make_table(w: Workload, device, seed: int = 0, chunk_rows: int = 1 << 22):
    """Value table [N, m] on ``device``: fp32 N(0, 0.02^2), cast with RNE for bf16."""
    import torch

    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    t = torch.empty((w.N, w.m), dtype=dt, device=device)
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    for s in range(0, w.N, chunk_rows):
        e = min(w.N, s + chunk_rows)
        t[s:e] = (torch.randn((e - s, w.m), generator=g, device=device, dtype=torch.float32) * TABLE_STD).to(dt)
    return t


def grad_out(w: Workload, device, seed: int = 0):
    """Upstream gradient [B, H, m] fp32 ~ N(0, 1) on ``device``."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed + 1)
    return torch.randn((w.B, w.H, w.m), generator=g, device=device, dtype=torch.float32)
