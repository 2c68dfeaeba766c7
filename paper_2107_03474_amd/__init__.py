"""LRAM lattice lookup on AMD Instinct MI355X -- Python binding of liblram.so.

Goucher & Troll, "Differentiable Random Access Memory using Lattices": the
lookup phi of Sec. 2.2 over Lambda = 2*E8 (Sec. 2.4) with the kernel of Sec. 2.5,
truncated to the closest 32 points found by the symmetry reduction of Sec. 2.6,
and its backward.

This module only marshals torch tensors (device memory) and the current HIP
stream into the C ABI declared in ``include/lram.h``; every step of the lookup
runs in the library's HIP kernels.  There is no fallback: if the library is not
built, or a call is made without a GPU, it raises.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import NamedTuple, Optional, Sequence, Tuple

import numpy as np
import torch  # noqa: F401  -- loads the HIP runtime liblram.so must share

__all__ = ["neighbors", "forward", "backward", "backward_workspace_bytes", "lookup", "LramLookup",
           "library_path", "load", "LramError", "F32", "BF16", "SCATTER_ATOMIC", "SCATTER_SORTED",
           "SCATTER_MERGED", "SCATTER_AUTO", "resolved_mode", "NB",
           "theta_coords", "theta_forward", "theta_backward", "ThetaLookup", "theta", "ALL", "MAX_SUPPORT",
           "list_width", "access_histogram", "access_stats", "sparse_adam", "SparseAdam", "Lists", "new_lists",
           "mark_touched",
           "order", "order_layout", "order_view", "backward_noalloc"]

NB = 32
F32, BF16 = 0, 1
SCATTER_ATOMIC, SCATTER_SORTED, SCATTER_MERGED, SCATTER_AUTO = 0, 1, 2, 3
_MODE_NAMES = {"atomic": SCATTER_ATOMIC, "sorted": SCATTER_SORTED, "merged": SCATTER_MERGED, "auto": SCATTER_AUTO}
_MODES = {**_MODE_NAMES, **{v: v for v in _MODE_NAMES.values()}}

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_build", "liblram.so")
_lock = threading.Lock()
_lib = None


class LramError(RuntimeError):
    pass


def library_path() -> str:
    return _LIB_PATH


def load():
    """Load liblram.so (built in-tree by ``paper_2107_03474_amd.build``)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                raise LramError("liblram.so is not built (%s); run paper_2107_03474_amd/build.py" % _LIB_PATH)
            lib = ctypes.CDLL(_LIB_PATH)
            P, I64, I32, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int
            lib.lram_version.restype = I
            lib.lram_strerror.argtypes = [I]
            lib.lram_strerror.restype = ctypes.c_char_p
            lib.lram_last_hip_error.restype = I
            lib.lram_neighbors.argtypes = [P, I64, I64, P, P, P, P, P]
            lib.lram_neighbors.restype = I
            lib.lram_forward.argtypes = [P, I64, I64, P, P, I, I64, I32, P, P, ctypes.c_size_t, P, P, P, P]
            lib.lram_forward.restype = I
            SZP = ctypes.POINTER(ctypes.c_size_t)
            lib.lram_order_bytes.argtypes = [I64, I64, SZP, SZP, SZP]
            lib.lram_order_bytes.restype = I
            lib.lram_order.argtypes = [P, I64, I64, P, P, ctypes.c_size_t, P]
            lib.lram_order.restype = I
            lib.lram_backward_workspace_bytes.argtypes = [I64, I64, I32, I, ctypes.POINTER(ctypes.c_size_t)]
            lib.lram_backward_workspace_bytes.restype = I
            lib.lram_scatter_mode_resolved.argtypes = [I64, I64, I, ctypes.POINTER(ctypes.c_int)]
            lib.lram_scatter_mode_resolved.restype = I
            lib.lram_backward.argtypes = [P, I64, I64, P, P, I, I64, I32, P, P, P, P, ctypes.c_size_t, P, P, P, I, P,
                                          ctypes.c_size_t, P]
            lib.lram_backward.restype = I
            lib.lram_backward_noalloc.argtypes = [P, I64, I64, P, P, I, I64, I32, P, P, P, I, P]
            lib.lram_backward_noalloc.restype = I
            lib.lram_neighbors_k.argtypes = [P, I64, I64, P, I32, P, P, P, P]
            lib.lram_neighbors_k.restype = I
            lib.lram_forward_k.argtypes = [P, I64, I64, P, P, I, I64, I32, I32, P, P]
            lib.lram_forward_k.restype = I
            lib.lram_backward_k.argtypes = [P, I64, I64, P, P, I, I64, I32, I32, P, P, P, I, P, ctypes.c_size_t,
                                            P]
            lib.lram_backward_k.restype = I
            lib.lram_access_histogram.argtypes = [P, I64, I64, P, P, P]
            lib.lram_access_histogram.restype = I
            lib.lram_access_stats.argtypes = [P, I64, P, P]
            lib.lram_access_stats.restype = I
            lib.lram_sparse_adam.argtypes = [P, I, I64, I32, P, P, P, I64, ctypes.c_double, ctypes.c_double,
                                             ctypes.c_double, ctypes.c_double, P]
            lib.lram_sparse_adam.restype = I
            lib.lram_mark_touched.argtypes = [P, I64, I64, P, P, P]
            lib.lram_mark_touched.restype = I
            lib.lram_sparse_adam_touched.argtypes = [P, I, I64, I32, P, P, P, P, I64, ctypes.c_double,
                                                     ctypes.c_double, ctypes.c_double, ctypes.c_double, P]
            lib.lram_sparse_adam_touched.restype = I
            lib.lram_theta_coords.argtypes = [P, I64, I64, P, P, P, P]
            lib.lram_theta_coords.restype = I
            lib.lram_theta_forward.argtypes = [P, I64, I64, P, P, I, I64, I32, P, P]
            lib.lram_theta_forward.restype = I
            lib.lram_theta_backward.argtypes = [P, I64, I64, P, P, I, I64, I32, P, P, P, I, P, ctypes.c_size_t, P]
            lib.lram_theta_backward.restype = I
            _lib = lib
    return _lib


def _check(rc: int):
    if rc != 0:
        lib = load()
        msg = lib.lram_strerror(rc).decode()
        if rc == 6:
            msg += " (hipError %d)" % lib.lram_last_hip_error()
        raise LramError(msg)


def _K(K: Sequence[int]):
    k = [int(v) for v in K]
    if len(k) != 8:
        raise LramError("K must have 8 entries")
    return (ctypes.c_int32 * 8)(*k)


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype=None, shape=None, like: Optional[torch.Tensor] = None):
    """Device pointer of t after checking what the kernels assume of it: a
    contiguous GPU tensor (on like's device), of the given dtype and shape --
    the C ABI takes raw pointers and cannot see a buffer's size."""
    if not t.is_cuda:
        raise LramError("%s must be a GPU tensor" % name)
    if like is not None and t.device != like.device:
        raise LramError("%s is on %s, expected %s" % (name, t.device, like.device))
    if not t.is_contiguous():
        raise LramError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise LramError("%s must be %s" % (name, dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise LramError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    return ctypes.c_void_p(t.data_ptr())


def _table_shape(table: torch.Tensor) -> Tuple[int, int]:
    if table.dim() != 2:
        raise LramError("table must be [N, m]")
    return table.shape[0], table.shape[1]


def _workspace(ws: Optional[torch.Tensor], like: torch.Tensor):
    """(pointer, size in bytes) of a backward workspace, (None, 0) for none."""
    if ws is None:
        return None, 0
    return _dev(ws, "workspace", like=like), ws.numel() * ws.element_size()


def _table_dtype(table: torch.Tensor) -> int:
    if table.dtype == torch.float32:
        return F32
    if table.dtype == torch.bfloat16:
        return BF16
    raise LramError("table must be float32 or bfloat16")


def _bh(q: torch.Tensor, last: int = 8, name: str = "q") -> Tuple[int, int]:
    if q.dim() not in (2, 3) or q.shape[-1] != last:
        raise LramError("%s must be [B, H, %d] or [L, %d]" % (name, last, last))
    if q.dim() == 2:
        return q.shape[0], 1
    return q.shape[0], q.shape[1]


ALL = 0             # k of the untruncated lookup (every point of the support)
MAX_SUPPORT = 256   # list width of the untruncated lookup


def list_width(k: int) -> int:
    return MAX_SUPPORT if k == ALL else int(k)


def neighbors(q: torch.Tensor, K: Sequence[int], want_d2: bool = True, k: int = NB):
    """Neighbour lists: (slot int32, w fp32, d2 fp32 or None), each [..., width]
    with width = k (16, 32, 64) or MAX_SUPPORT for k = ALL."""
    lib = load()
    B, H = _bh(q)
    lead = q.shape[:-1]
    wd = list_width(k)
    slot = torch.empty(lead + (wd,), dtype=torch.int32, device=q.device)
    w = torch.empty(lead + (wd,), dtype=torch.float32, device=q.device)
    d2 = torch.empty(lead + (wd,), dtype=torch.float32, device=q.device) if want_d2 else None
    _check(lib.lram_neighbors_k(_dev(q, "q", torch.float32), B, H, _K(K), int(k), _dev(slot, "slot"), _dev(w, "w"),
                                _dev(d2, "d2") if d2 is not None else None, _stream(q)))
    return slot, w, d2


class Lists(NamedTuple):
    """Neighbour lists saved by ``forward`` for ``backward`` (each [..., 32]):
    location (-1 padding), recipe weight, and the point's code in its query's
    fundamental-region frame."""
    slot: torch.Tensor
    w: torch.Tensor
    code: torch.Tensor


def new_lists(q: torch.Tensor) -> Lists:
    """Uninitialised saved-list buffers for the lookups of q [..., 8]."""
    lead = q.shape[:-1] + (NB,)
    return Lists(torch.empty(lead, dtype=torch.int32, device=q.device),
                 torch.empty(lead, dtype=torch.float32, device=q.device),
                 torch.empty(lead, dtype=torch.int32, device=q.device))


def _lists(nl: Optional[Lists], q: torch.Tensor):
    if nl is None:
        return None, None, None
    lead = q.shape[:-1] + (NB,)
    return (_dev(nl.slot, "lists.slot", torch.int32, lead, like=q), _dev(nl.w, "lists.w", torch.float32, lead, like=q),
            _dev(nl.code, "lists.code", torch.int32, lead, like=q))


def order_layout(B: int, H: int) -> Tuple[int, int, int]:
    """(bytes, keys offset, perm offset) of an order buffer for B*H lookups."""
    lib = load()
    n, ko, po = ctypes.c_size_t(0), ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(lib.lram_order_bytes(B, H, ctypes.byref(n), ctypes.byref(ko), ctypes.byref(po)))
    return n.value, ko.value, po.value


def order(q: torch.Tensor, K: Sequence[int], buf: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The lookups of q sorted by the location of their closest lattice point
    (lram_order): a uint8 device buffer to pass as ``order=`` to forward and
    backward (and usable as the merged scatter's workspace)."""
    lib = load()
    B, H = _bh(q)
    nbytes = order_layout(B, H)[0]
    if buf is None:
        buf = torch.empty(nbytes, dtype=torch.uint8, device=q.device)
    _check(lib.lram_order(_dev(q, "q", torch.float32), B, H, _K(K), _dev(buf, "order", torch.uint8, like=q),
                          buf.numel(), _stream(q)))
    return buf


def order_view(buf: torch.Tensor, L: int):
    """(shared count [1], keys [L], perm [L]) int32 views of an order buffer
    (uint32 values; L < 2^31 keeps them non-negative)."""
    _, ko, po = order_layout(L, 1)
    w = buf.view(torch.int32)
    return w[:1], w[ko // 4:ko // 4 + L], w[po // 4:po // 4 + L]


def _order(buf: Optional[torch.Tensor], q: torch.Tensor):
    if buf is None:
        return None, 0
    return _dev(buf, "order", torch.uint8, like=q), buf.numel()


def forward(q: torch.Tensor, table: torch.Tensor, K: Sequence[int], out: Optional[torch.Tensor] = None,
            k: int = NB, order: Optional[torch.Tensor] = None, lists: Optional[Lists] = None):
    """phi(q) over the closest k points (k = ALL: the whole support): [..., m] in the table dtype.
    k = 32 only: ``order`` (from ``order()``) visits the lookups in that order;
    ``lists`` (from ``new_lists``) receives the neighbour lists for ``backward``."""
    lib = load()
    B, H = _bh(q)
    N, m = _table_shape(table)
    if out is None:
        out = torch.empty(q.shape[:-1] + (m,), dtype=table.dtype, device=q.device)
    args = (_dev(q, "q", torch.float32), B, H, _K(K), _dev(table, "table", like=q), _table_dtype(table), N, m)
    o = _dev(out, "out", table.dtype, q.shape[:-1] + (m,), like=q)
    if k == NB:
        _check(lib.lram_forward(*args, o, *_order(order, q), *_lists(lists, q), _stream(q)))
    else:
        if order is not None or lists is not None:
            raise LramError("order and saved lists are offered for k = 32 only")
        _check(lib.lram_forward_k(*args, int(k), o, _stream(q)))
    return out


def resolved_mode(B: int, H: int, mode="auto") -> str:
    """Name of the scatter mode lram_backward runs for B*H lookups given ``mode``."""
    lib = load()
    r = ctypes.c_int(-1)
    _check(lib.lram_scatter_mode_resolved(B, H, _MODES[mode], ctypes.byref(r)))
    return {v: k for k, v in _MODE_NAMES.items()}[r.value]


def backward_workspace_bytes(B: int, H: int, m: int, mode="auto") -> int:
    lib = load()
    n = ctypes.c_size_t(0)
    _check(lib.lram_backward_workspace_bytes(B, H, m, _MODES[mode], ctypes.byref(n)))
    return n.value


def backward(q: torch.Tensor, table: torch.Tensor, K: Sequence[int], grad_out: torch.Tensor,
             grad_table: Optional[torch.Tensor] = None, want_grad_q: bool = True, mode="auto",
             workspace: Optional[torch.Tensor] = None, grad_q: Optional[torch.Tensor] = None, k: int = NB,
             order: Optional[torch.Tensor] = None, lists: Optional[Lists] = None):
    """Gradients: grad_table [N, m] fp32 is ACCUMULATED into (allocated zeroed if None,
    pass False to skip), grad_q [..., 8] fp32 (None unless want_grad_q; written into
    ``grad_q`` when given).  k != 32 (variable k / ALL) takes the atomic and
    merged scatters (and "auto"), not the sorted one.  k = 32 only: ``order``
    (from ``order()``) replaces the merged scatter's sort; ``lists`` (filled by
    ``forward``) replace the neighbour search."""
    lib = load()
    B, H = _bh(q)
    N, m = _table_shape(table)
    if grad_table is None:
        grad_table = torch.zeros((N, m), dtype=torch.float32, device=q.device)
    gq = None
    if want_grad_q:
        gq = grad_q if grad_q is not None else torch.empty(q.shape, dtype=torch.float32, device=q.device)
    head = (_dev(q, "q", torch.float32), B, H, _K(K), _dev(table, "table", like=q), _table_dtype(table), N, m)
    grads = (_dev(grad_out, "grad_out", torch.float32, q.shape[:-1] + (m,), like=q),
             _dev(grad_table, "grad_table", torch.float32, (N, m), like=q) if grad_table is not False else None,
             _dev(gq, "grad_q", torch.float32, q.shape, like=q) if gq is not None else None)
    mode_i = _MODES[mode]
    ws_bytes = backward_workspace_bytes(B, H, m, mode_i)
    merged_with_order = order is not None and resolved_mode(B, H, mode_i) == "merged"
    if ws_bytes and workspace is None and not merged_with_order:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    if k != NB:
        if order is not None or lists is not None:
            raise LramError("order and saved lists are offered for k = 32 only")
        _check(lib.lram_backward_k(*head, int(k), *grads, mode_i, *_workspace(workspace, q), _stream(q)))
    else:
        _check(lib.lram_backward(*head, *grads, *_order(order, q), *_lists(lists, q), mode_i,
                                 *_workspace(workspace, q), _stream(q)))
    return (grad_table if grad_table is not False else None), gq


def backward_noalloc(q: torch.Tensor, table: torch.Tensor, K: Sequence[int], grad_out: torch.Tensor,
                     grad_table: torch.Tensor, grad_q: Optional[torch.Tensor] = None, mode="auto"):
    """lram_backward_noalloc: ``backward`` whose scatter workspace is the library's
    static per-GPU array (nothing allocated by the call).  grad_table [N, m] fp32
    is accumulated into, grad_q [..., 8] fp32 (nullable) overwritten."""
    lib = load()
    B, H = _bh(q)
    N, m = _table_shape(table)
    _check(lib.lram_backward_noalloc(
        _dev(q, "q", torch.float32), B, H, _K(K), _dev(table, "table", like=q), _table_dtype(table), N, m,
        _dev(grad_out, "grad_out", torch.float32, q.shape[:-1] + (m,), like=q),
        _dev(grad_table, "grad_table", torch.float32, (N, m), like=q),
        _dev(grad_q, "grad_q", torch.float32, q.shape, like=q) if grad_q is not None else None, _MODES[mode],
        _stream(q)))


class LramLookup(torch.autograd.Function):
    """Autograd wrapper (Sec. 2.6): forward phi(q); backward gives dq and a dense
    dtable.  save_lists: the forward keeps the neighbour lists (384 bytes per
    lookup) and the backward reuses them instead of searching again."""

    @staticmethod
    def forward(ctx, q, table, K, mode, save_lists):
        q, table = q.contiguous(), table.contiguous()
        ctx.K = tuple(int(k) for k in K)
        ctx.mode = mode
        nl = new_lists(q) if save_lists else None
        out = forward(q, table, ctx.K, lists=nl)
        ctx.save_for_backward(q, table, *(nl if nl is not None else ()))
        return out

    @staticmethod
    def backward(ctx, g):
        q, table, *saved = ctx.saved_tensors
        g32 = g.contiguous().to(torch.float32)
        gt, gq = backward(q, table, ctx.K, g32, grad_table=None if ctx.needs_input_grad[1] else False,
                          want_grad_q=ctx.needs_input_grad[0], mode=ctx.mode,
                          lists=Lists(*saved) if saved else None)
        return gq, (gt.to(table.dtype) if gt is not None else None), None, None, None


def lookup(q: torch.Tensor, table: torch.Tensor, K: Sequence[int], mode="auto", save_lists: bool = False) -> torch.Tensor:
    return LramLookup.apply(q, table, tuple(K), mode, bool(save_lists))


# ---------------------------------------------------------------------------
# Activation layer (Sec. 2.3): z [..., 16] = 8 complex numbers (Re, Im) per head.

def theta_coords(z: torch.Tensor, K: Sequence[int]):
    """(q [..., 8] fp32, s [...] fp32): torus coordinates and output scale of theta."""
    lib = load()
    B, H = _bh(z, 16, "z")
    q = torch.empty(z.shape[:-1] + (8,), dtype=torch.float32, device=z.device)
    sc = torch.empty(z.shape[:-1], dtype=torch.float32, device=z.device)
    _check(lib.lram_theta_coords(_dev(z, "z", torch.float32), B, H, _K(K), _dev(q, "q"), _dev(sc, "s"), _stream(z)))
    return q, sc


def theta_forward(z: torch.Tensor, table: torch.Tensor, K: Sequence[int], out: Optional[torch.Tensor] = None):
    """theta(z) = (sum 1/|z_i|)^-1 phi((K_i / 2 pi) arg z_i): [..., m] in the table dtype."""
    lib = load()
    B, H = _bh(z, 16, "z")
    N, m = _table_shape(table)
    if out is None:
        out = torch.empty(z.shape[:-1] + (m,), dtype=table.dtype, device=z.device)
    _check(lib.lram_theta_forward(_dev(z, "z", torch.float32), B, H, _K(K), _dev(table, "table", like=z),
                                  _table_dtype(table), N, m, _dev(out, "out", table.dtype, z.shape[:-1] + (m,), like=z),
                                  _stream(z)))
    return out


def theta_backward(z: torch.Tensor, table: torch.Tensor, K: Sequence[int], grad_out: torch.Tensor,
                   grad_table: Optional[torch.Tensor] = None, want_grad_z: bool = True, mode="auto",
                   workspace: Optional[torch.Tensor] = None, grad_z: Optional[torch.Tensor] = None):
    """Gradients of <grad_out, theta(z)>: grad_table [N, m] fp32 ACCUMULATED into
    (allocated zeroed if None, False to skip), grad_z [..., 16] fp32."""
    lib = load()
    B, H = _bh(z, 16, "z")
    N, m = _table_shape(table)
    if grad_table is None:
        grad_table = torch.zeros((N, m), dtype=torch.float32, device=z.device)
    gz = None
    if want_grad_z:
        gz = grad_z if grad_z is not None else torch.empty(z.shape, dtype=torch.float32, device=z.device)
    mode_i = _MODES[mode]
    ws_bytes = backward_workspace_bytes(B, H, m, mode_i)
    if ws_bytes and workspace is None:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=z.device)
    _check(lib.lram_theta_backward(
        _dev(z, "z", torch.float32), B, H, _K(K), _dev(table, "table", like=z), _table_dtype(table), N, m,
        _dev(grad_out, "grad_out", torch.float32, z.shape[:-1] + (m,), like=z),
        _dev(grad_table, "grad_table", torch.float32, (N, m), like=z) if grad_table is not False else None,
        _dev(gz, "grad_z", torch.float32, z.shape, like=z) if gz is not None else None, mode_i,
        *_workspace(workspace, z), _stream(z)))
    return (grad_table if grad_table is not False else None), gz


class ThetaLookup(torch.autograd.Function):
    """Autograd wrapper of the activation layer + lookup: dz and a dense dtable."""

    @staticmethod
    def forward(ctx, z, table, K, mode):
        z, table = z.contiguous(), table.contiguous()
        ctx.save_for_backward(z, table)
        ctx.K = tuple(int(k) for k in K)
        ctx.mode = mode
        return theta_forward(z, table, ctx.K)

    @staticmethod
    def backward(ctx, g):
        z, table = ctx.saved_tensors
        g32 = g.contiguous().to(torch.float32)
        gt, gz = theta_backward(z, table, ctx.K, g32, grad_table=None if ctx.needs_input_grad[1] else False,
                                want_grad_z=ctx.needs_input_grad[0], mode=ctx.mode)
        return gz, (gt.to(table.dtype) if gt is not None else None), None, None


def theta(z: torch.Tensor, table: torch.Tensor, K: Sequence[int], mode="auto") -> torch.Tensor:
    return ThetaLookup.apply(z, table, tuple(K), mode)


# ---------------------------------------------------------------------------
# Training-side companions: access statistics and the sparse Adam step.

def access_histogram(q: torch.Tensor, K: Sequence[int], hist: Optional[torch.Tensor] = None) -> torch.Tensor:
    """hist [N] fp32 += the kernel weights of every (lookup, neighbour) pair at its location."""
    lib = load()
    B, H = _bh(q)
    N = int(np.prod([int(k) for k in K]))
    if hist is None:
        hist = torch.zeros(N, dtype=torch.float32, device=q.device)
    _check(lib.lram_access_histogram(_dev(q, "q", torch.float32), B, H, _K(K),
                                     _dev(hist, "hist", torch.float32, (N,), like=q), _stream(q)))
    return hist


def access_stats(hist: torch.Tensor) -> dict:
    """{used: fraction of locations accessed, kl: KL(access distribution || uniform),
    total: summed weight, count: locations accessed} (synchronises to read them)."""
    lib = load()
    out = torch.empty(4, dtype=torch.float64, device=hist.device)
    if hist.dim() != 1:
        raise LramError("hist must be [N]")
    _check(lib.lram_access_stats(_dev(hist, "hist", torch.float32), hist.numel(), _dev(out, "out"), _stream(hist)))
    v = out.cpu().tolist()
    return {"used": v[0], "kl": v[1], "total": v[2], "count": int(round(v[3]))}


def mark_touched(q: torch.Tensor, K: Sequence[int], touched: Optional[torch.Tensor] = None) -> torch.Tensor:
    """touched [N] uint8: set to 1 at every location in the closest-32 lists of
    the lookups of q (allocated zeroed if None; other entries unchanged)."""
    lib = load()
    B, H = _bh(q)
    N = int(np.prod([int(k) for k in K]))
    if touched is None:
        touched = torch.zeros(N, dtype=torch.uint8, device=q.device)
    _check(lib.lram_mark_touched(_dev(q, "q", torch.float32), B, H, _K(K),
                                 _dev(touched, "touched", torch.uint8, (N,), like=q), _stream(q)))
    return touched


def sparse_adam(table: torch.Tensor, grad: torch.Tensor, exp_avg: torch.Tensor, exp_avg_sq: torch.Tensor,
                step: int, lr: float = 1e-3, betas=(0.9, 0.999), eps: float = 1e-8,
                touched: Optional[torch.Tensor] = None):
    """One Adam step on the rows of ``table`` whose ``grad`` row is not all zero
    (in place; those grad rows are cleared).  With ``touched`` (from
    ``mark_touched``) only the flagged rows are visited and the flags cleared."""
    lib = load()
    N, m = _table_shape(table)
    f32 = torch.float32
    args = (_dev(table, "table"), _table_dtype(table), N, m, _dev(grad, "grad", f32, (N, m), like=table),
            _dev(exp_avg, "exp_avg", f32, (N, m), like=table), _dev(exp_avg_sq, "exp_avg_sq", f32, (N, m), like=table))
    hyper = (int(step), float(lr), float(betas[0]), float(betas[1]), float(eps), _stream(table))
    if touched is None:
        _check(lib.lram_sparse_adam(*args, *hyper))
    else:
        _check(lib.lram_sparse_adam_touched(*args, _dev(touched, "touched", torch.uint8, (N,), like=table), *hyper))


class SparseAdam:
    """Adam state for one lattice memory table (the memory parameters of
    Sec. 3.2, learning rate 1e-3): call ``step(grad)`` with the accumulated
    fp32 gradient table; untouched rows keep value and moments."""

    def __init__(self, table: torch.Tensor, lr: float = 1e-3, betas=(0.9, 0.999), eps: float = 1e-8):
        self.table, self.lr, self.betas, self.eps, self.t = table, lr, betas, eps, 0
        self.exp_avg = torch.zeros(table.shape, dtype=torch.float32, device=table.device)
        self.exp_avg_sq = torch.zeros(table.shape, dtype=torch.float32, device=table.device)

    def step(self, grad: torch.Tensor, touched: Optional[torch.Tensor] = None):
        """touched: flags from ``mark_touched`` for the step's lookups (the step
        then visits only those rows)."""
        self.t += 1
        sparse_adam(self.table, grad, self.exp_avg, self.exp_avg_sq, self.t, self.lr, self.betas, self.eps,
                    touched=touched)
