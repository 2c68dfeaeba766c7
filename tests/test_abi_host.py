"""Host-side checks of the C ABI: the library loads, exports every entry point
declared in include/lram.h, and rejects bad arguments before launching anything.
No GPU is needed: every call here fails (or returns) in host validation."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2107_03474_amd as lram

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lram.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(lram_[a-z_0-9]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def lib():
    return lram.load()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert {"lram_forward", "lram_backward", "lram_neighbors", "lram_backward_workspace_bytes",
            "lram_strerror", "lram_version", "lram_last_hip_error"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", lram.library_path()], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (lram_[a-z_0-9]+)", out))
    assert set(names) <= exported, set(names) - exported
    for n in names:
        assert hasattr(lib, n)


def test_version_and_strerror(lib):
    assert lib.lram_version() >= 100
    for rc in range(7):
        assert len(lib.lram_strerror(rc)) > 0
    assert b"unknown" in lib.lram_strerror(99)


K4 = (ctypes.c_int32 * 8)(*([4] * 8))
FAKE = ctypes.c_void_p(0x10000)      # never dereferenced: validation fails first
FAKE_MIS = ctypes.c_void_p(0x10004)  # misaligned


def _fwd(lib, q=FAKE, B=4, H=1, K=K4, table=FAKE, dtype=0, N=4 ** 8, m=32, out=FAKE, order=None, ob=0, slot=None,
         w=None, code=None):
    return lib.lram_forward(q, B, H, K, table, dtype, N, m, out, order, ob, slot, w, code, None)


def test_forward_validation(lib):
    assert _fwd(lib, K=(ctypes.c_int32 * 8)(*([3] + [4] * 7))) == 2          # odd K
    assert _fwd(lib, K=(ctypes.c_int32 * 8)(*([0] + [4] * 7))) == 2          # K < 2
    assert _fwd(lib, K=(ctypes.c_int32 * 8)(*([16] * 8))) == 2                # N >= 2^31
    assert _fwd(lib, N=12345) == 2                                            # N != prod K
    big = (ctypes.c_int32 * 8)(*([8194, 2, 2, 2, 2, 2, 2, 2]))
    assert _fwd(lib, K=big, N=8194 * 128) == 2                                # K_i > 8192
    assert _fwd(lib, dtype=7) == 3
    assert _fwd(lib, m=48) == 3
    assert _fwd(lib, q=None) == 1
    assert _fwd(lib, q=FAKE_MIS) == 1
    assert _fwd(lib, table=None) == 1
    assert _fwd(lib, out=None) == 1
    assert _fwd(lib, B=-1) == 1
    assert _fwd(lib, B=1 << 31) == 1                                          # L >= 2^31 lookups
    assert _fwd(lib, B=1 << 16, H=1 << 15) == 1
    assert _fwd(lib, B=1 << 62, H=4) == 1                                      # B*H overflows int64
    assert _fwd(lib, q=None, table=None, out=None, B=0) == 0                  # empty: no-op
    assert _fwd(lib, q=None, table=None, out=None, H=0) == 0


def test_order_and_saved_list_validation(lib):
    """Order buffers are 256-byte aligned and large enough for the call's
    lookups; saved lists come as all three arrays or none, 4-byte aligned."""
    n, ko, po = ctypes.c_size_t(0), ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert lib.lram_order_bytes(1000, 3, ctypes.byref(n), ctypes.byref(ko), ctypes.byref(po)) == 0
    assert ko.value == 256 and po.value == 256 + 12032 and n.value >= po.value + 12000
    assert lib.lram_order_bytes(-1, 3, ctypes.byref(n), None, None) == 1
    assert lib.lram_order_bytes(1 << 31, 1, ctypes.byref(n), None, None) == 1
    need = ctypes.c_size_t(0)
    assert lib.lram_order_bytes(4, 1, ctypes.byref(need), None, None) == 0
    ORD = ctypes.c_void_p(0x20000)
    assert lib.lram_order(FAKE, 4, 1, K4, None, need.value, None) == 1
    assert lib.lram_order(FAKE, 4, 1, K4, ORD, need.value - 1, None) == 1                 # undersized
    assert lib.lram_order(FAKE, 4, 1, K4, ctypes.c_void_p(0x20010), need.value, None) == 1  # misaligned
    assert lib.lram_order(FAKE, 4, 1, (ctypes.c_int32 * 8)(*([3] * 8)), ORD, need.value, None) == 2
    assert lib.lram_order(None, 0, 1, K4, ORD, need.value, None) == 0
    assert _fwd(lib, order=ORD, ob=need.value - 256) == 1
    assert _fwd(lib, order=ctypes.c_void_p(0x20080), ob=need.value) == 1
    assert _fwd(lib, slot=FAKE, w=FAKE) == 1                                   # lists incomplete
    assert _fwd(lib, slot=FAKE, w=FAKE, code=ctypes.c_void_p(0x10002)) == 1    # misaligned
    assert _fwd(lib, slot=FAKE, code=FAKE) == 1

    def bwd(order=None, ob=0, slot=None, w=None, code=None):
        return lib.lram_backward(FAKE, 4, 1, K4, FAKE, 0, 4 ** 8, 32, FAKE, FAKE, FAKE, order, ob, slot, w, code, 2,
                                 None, 0, None)

    assert bwd(slot=FAKE) == 1
    assert bwd(order=ORD, ob=need.value - 1) == 1
    assert bwd() == 4                                  # merged without an order needs a workspace


def test_neighbors_validation(lib):
    assert lib.lram_neighbors(FAKE, 4, 1, (ctypes.c_int32 * 8)(*([5] * 8)), FAKE, FAKE, None, None) == 2
    assert lib.lram_neighbors(FAKE, 4, 1, K4, None, FAKE, None, None) == 1
    assert lib.lram_neighbors(None, 0, 7, K4, None, None, None, None) == 0
    odd = ctypes.c_void_p(0x10002)  # not 4-byte aligned
    assert lib.lram_neighbors(FAKE, 4, 1, K4, odd, FAKE, None, None) == 1
    assert lib.lram_neighbors(FAKE, 4, 1, K4, FAKE, odd, None, None) == 1
    assert lib.lram_neighbors(FAKE, 4, 1, K4, FAKE, FAKE, odd, None) == 1
    assert lib.lram_neighbors_k(FAKE, 4, 1, K4, 16, FAKE, FAKE, odd, None) == 1


def test_backward_validation(lib):
    def bwd(grad_out=FAKE, gt=FAKE, gq=FAKE, mode=0, K=K4, B=4, ws=None, wsb=0):
        return lib.lram_backward(FAKE, B, 1, K, FAKE, 0, 4 ** 8, 32, grad_out, gt, gq, None, 0, None, None, None, mode,
                                 ws, wsb, None)

    assert bwd(mode=9) == 5
    assert bwd(grad_out=None) == 1
    assert bwd(gt=None, gq=None) == 1
    assert bwd(K=(ctypes.c_int32 * 8)(*([4] * 7 + [7]))) == 2
    assert bwd(B=0, grad_out=None) == 0
    n = ctypes.c_size_t(123)
    assert lib.lram_backward_workspace_bytes(4, 1, 32, 0, ctypes.byref(n)) == 0 and n.value == 0
    assert lib.lram_backward_workspace_bytes(4, 1, 32, 9, ctypes.byref(n)) == 5
    assert lib.lram_backward_workspace_bytes(4, 1, 32, 1, ctypes.byref(n)) == 0 and n.value >= 4 * 32 * 24
    assert bwd(mode=1, ws=None) == 4  # sorted mode without a workspace
    assert lib.lram_backward_workspace_bytes(4, 1, 32, 2, ctypes.byref(n)) == 0 and n.value >= 4 * 24
    assert bwd(mode=2, ws=None) == 4  # merged mode without a workspace
    assert bwd(mode=2, ws=FAKE_MIS, wsb=1 << 20) == 4  # misaligned workspace
    assert lib.lram_backward_workspace_bytes(4, 1, 48, 0, ctypes.byref(n)) == 3


def test_theta_validation(lib):
    K7 = (ctypes.c_int32 * 8)(*([4] * 7 + [7]))
    assert lib.lram_theta_forward(FAKE, 4, 1, K7, FAKE, 0, 4 ** 8, 32, FAKE, None) == 2
    assert lib.lram_theta_forward(None, 4, 1, K4, FAKE, 0, 4 ** 8, 32, FAKE, None) == 1
    assert lib.lram_theta_forward(FAKE_MIS, 4, 1, K4, FAKE, 0, 4 ** 8, 32, FAKE, None) == 1
    assert lib.lram_theta_forward(FAKE, 4, 1, K4, FAKE, 0, 4 ** 8, 40, FAKE, None) == 3
    assert lib.lram_theta_forward(None, 0, 3, K4, None, 0, 4 ** 8, 32, None, None) == 0
    assert lib.lram_theta_coords(FAKE, 4, 1, K4, None, None, None) == 1
    assert lib.lram_theta_coords(None, 0, 1, K4, None, None, None) == 0
    assert lib.lram_theta_coords(FAKE, 4, 1, K4, FAKE_MIS, None, None) == 1   # q is written as 16-byte vectors
    assert lib.lram_theta_coords(FAKE, 4, 1, K4, FAKE, ctypes.c_void_p(0x10001), None) == 1
    assert lib.lram_theta_backward(FAKE, 4, 1, K4, FAKE, 0, 4 ** 8, 32, FAKE, None, None, 0, None, 0, None) == 1
    assert lib.lram_theta_backward(FAKE, 4, 1, K4, FAKE, 0, 4 ** 8, 32, FAKE, FAKE, FAKE, 7, None, 0, None) == 5
    assert lib.lram_theta_backward(FAKE, 4, 1, K4, FAKE, 0, 4 ** 8, 32, FAKE, FAKE, FAKE, 2, None, 0, None) == 4


def test_variable_k_validation(lib):
    assert lib.lram_forward_k(FAKE, 4, 1, K4, FAKE, 0, 4 ** 8, 32, 48, FAKE, None) == 1   # k not offered
    assert lib.lram_forward_k(FAKE, 4, 1, K4, FAKE, 0, 4 ** 8, 32, -1, FAKE, None) == 1
    assert lib.lram_neighbors_k(FAKE, 4, 1, K4, 128, FAKE, FAKE, None, None) == 1
    assert lib.lram_neighbors_k(FAKE, 4, 1, (ctypes.c_int32 * 8)(*([5] * 8)), 0, FAKE, FAKE, None, None) == 2
    def bwd_k(k=16, m=32, grad_out=FAKE, mode=0, ws=None, wsb=0):
        return lib.lram_backward_k(FAKE, 4, 1, K4, FAKE, 0, 4 ** 8, m, k, grad_out, FAKE, FAKE, mode, ws, wsb, None)

    assert bwd_k(grad_out=None) == 1
    assert bwd_k(m=40) == 3
    assert bwd_k(k=48) == 1
    assert bwd_k(mode=1) == 5                      # the sorted scatter takes k = 32 only
    assert bwd_k(k=0, mode=1) == 5
    assert bwd_k(mode=2) == 4                      # merged without a workspace
    assert bwd_k(k=64, mode=2, ws=FAKE_MIS, wsb=1 << 20) == 4
    assert bwd_k(mode=7) == 5
    assert lib.lram_forward_k(None, 0, 1, K4, None, 0, 4 ** 8, 32, 0, None, None) == 0


def test_training_entry_points_validation(lib):
    lib.lram_sparse_adam.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_double,
                                     ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_void_p]
    ok = dict(table=FAKE, dtype=0, N=100, m=32, grad=FAKE, m1=FAKE, m2=FAKE, step=1, lr=1e-3, b1=0.9, b2=0.999,
              eps=1e-8)

    def adam(**kw):
        a = dict(ok, **kw)
        return lib.lram_sparse_adam(a["table"], a["dtype"], a["N"], a["m"], a["grad"], a["m1"], a["m2"], a["step"],
                                    a["lr"], a["b1"], a["b2"], a["eps"], None)

    assert adam(step=0) == 1
    assert adam(b1=1.0) == 1
    assert adam(b2=-0.1) == 1
    assert adam(lr=float("nan")) == 1
    assert adam(m=48) == 3
    assert adam(dtype=5) == 3
    assert adam(grad=None) == 1
    assert adam(m1=FAKE_MIS) == 1
    assert adam(N=0, table=None, grad=None, m1=None, m2=None) == 0
    assert lib.lram_access_stats(FAKE, 0, FAKE, None) == 1
    assert lib.lram_access_stats(FAKE, 10, None, None) == 1
    assert lib.lram_access_histogram(FAKE, 4, 1, K4, None, None) == 1
    assert lib.lram_access_histogram(None, 0, 1, K4, None, None) == 0
    assert lib.lram_access_histogram(FAKE, 4, 1, K4, ctypes.c_void_p(0x10002), None) == 1   # fp32 atomics
    assert lib.lram_access_stats(ctypes.c_void_p(0x10002), 10, FAKE, None) == 1


def test_auto_mode(lib):
    r = ctypes.c_int(-1)
    assert lib.lram_scatter_mode_resolved(4, 1, 3, ctypes.byref(r)) == 0 and r.value == 0        # small: atomic
    assert lib.lram_scatter_mode_resolved(8192, 16, 3, ctypes.byref(r)) == 0 and r.value == 2    # 131072: merged
    assert lib.lram_scatter_mode_resolved(8192, 16, 1, ctypes.byref(r)) == 0 and r.value == 1    # explicit kept
    assert lib.lram_scatter_mode_resolved(4, 1, 4, ctypes.byref(r)) == 5
    assert lib.lram_scatter_mode_resolved(-1, 1, 0, ctypes.byref(r)) == 1
    n = ctypes.c_size_t(1)
    assert lib.lram_backward_workspace_bytes(4, 1, 32, 3, ctypes.byref(n)) == 0 and n.value == 0
    assert lib.lram_backward_workspace_bytes(8192, 16, 32, 3, ctypes.byref(n)) == 0 and n.value >= 131072 * 16


def test_no_oracle_in_product():
    """The product package never imports or links the oracle."""
    pkg = os.path.join(ROOT, "paper_2107_03474_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h", ".inc")):
                txt = open(os.path.join(dirpath, f), errors="ignore").read()
                assert "oracle" not in txt.lower(), f
    out = subprocess.run(["ldd", lram.library_path()], capture_output=True, text=True).stdout
    assert "oracle" not in out
