"""Memory-augmented subnetwork (Sec. 3.1) on the lattice lookup.

y = W2 theta(BN(W1 x + b1)) + b2: a dense affine layer R^w -> R^w, batch
normalisation of the query vector (Sec. 4.1), the activation layer + lookup
of Sec. 2.3 with (n, m, h) = (8, 64, w/16) on one shared table (so theta maps
R^w to R^{4w}), and a dense affine layer R^{4w} -> R^w.  The dense layers and
the normalisation are library operations (GEMMs through the platform BLAS);
theta and the lookup run in liblram's kernels through ``ThetaLookup``.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import theta as _theta

M_VALUE = 64


class MemorySubnetwork(torch.nn.Module):
    def __init__(self, w: int, K: Sequence[int], table_dtype=torch.bfloat16, dtype=torch.float32,
                 table_std: float = 0.02, device="cuda", scatter: str = "auto",
                 table: Optional[torch.Tensor] = None):
        super().__init__()
        if w % 16:
            raise ValueError("w must be a multiple of 16 (h = w/16 heads of 8 complex numbers)")
        self.w, self.h, self.K, self.scatter = w, w // 16, tuple(int(k) for k in K), scatter
        N = int(np.prod(self.K))
        self.inp = torch.nn.Linear(w, w, device=device, dtype=dtype)
        self.bn = torch.nn.BatchNorm1d(w, device=device, dtype=dtype)
        self.out = torch.nn.Linear(self.h * M_VALUE, w, device=device, dtype=dtype)
        if table is not None:  # a shared, already initialised table [N, 64]
            if tuple(table.shape) != (N, M_VALUE):
                raise ValueError("table must be [prod K, 64]")
            self.table = torch.nn.Parameter(table, requires_grad=table.requires_grad)
            return
        t = torch.empty((N, M_VALUE), device=device, dtype=table_dtype)
        chunk = 1 << 22
        for s in range(0, N, chunk):
            t[s:s + chunk] = torch.randn((min(chunk, N - s), M_VALUE), device=device) * table_std
        self.table = torch.nn.Parameter(t)

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        T = x.shape[0]
        z = self.bn(self.inp(x)).float().reshape(T, self.h, 16).contiguous()
        th = _theta(z, self.table, self.K, self.scatter)          # [T, h, 64]
        return self.out(th.reshape(T, self.h * M_VALUE).to(self.out.weight.dtype))
