"""C-ABI checks that need no GPU: the library loads, exports every function
declared in include/acdc.h, and rejects bad arguments on the host before any
HIP call (so these run on a machine without a GPU)."""

import ctypes
import os
import re

import pytest

from paper_1511_05946_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "acdc.h")

OK, EINVAL, EUNSUP, EWS, EHIP = 0, -1, -2, -3, -4
PERM, RELU, CX = 1, 2, 4


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libacdc.so is not built (run __graft_entry__.build())")
    return _lib.lib()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(acdc_[a-z_]+)\s*\(", src)))


def test_header_declares_expected_entry_points():
    names = declared_functions()
    for n in ("acdc_forward", "acdc_backward", "acdc_backward_workspace_bytes", "acdc_prepare",
              "acdc_status_string", "acdc_last_hip_error", "acdc_supported"):
        assert n in names


def test_every_declared_symbol_is_exported(L):
    for n in declared_functions():
        assert hasattr(L, n), n
        assert n in _lib.SIGNATURES, f"binding lacks a signature for {n}"


def test_supported_widths(L):
    for N in (8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096, 8192, 9216, 16384):
        assert L.acdc_supported(N, 0) == 1
        assert L.acdc_supported(N, PERM | RELU) == 1
    for N in (8, 64, 1024, 4096, 8192):
        assert L.acdc_supported(N, CX | PERM) == 1
    for N in (0, 2, 4, 6, 12, 100, 1000, 3072, 32768):
        assert L.acdc_supported(N, 0) == 0
    assert L.acdc_supported(9216, CX) == 0
    assert L.acdc_supported(4096, CX | RELU) == 0
    assert L.acdc_supported(4096, 8) == 0


def test_status_strings(L):
    for rc in (OK, EINVAL, EUNSUP, EWS, EHIP, 99):
        assert isinstance(L.acdc_status_string(rc), bytes)
    assert L.acdc_status_string(OK) == b"ok"


def test_sizes(L):
    assert L.acdc_saved_bytes(8192, 4096, 12, PERM | RELU) == 11 * 8192 * 4096 * 4
    assert L.acdc_saved_bytes(10, 64, 1, 0) == 0
    assert L.acdc_saved_bytes(10, 64, 3, CX) == 2 * 10 * 64 * 8
    ws_saved = L.acdc_backward_workspace_bytes(8192, 4096, 12, PERM | RELU, 1)
    ws_recompute = L.acdc_backward_workspace_bytes(8192, 4096, 12, PERM | RELU, 0)
    assert ws_saved > 0 and ws_recompute >= ws_saved + 11 * 8192 * 4096 * 4
    assert L.acdc_forward_workspace_bytes(8192, 4096, 12, 0) > 0
    assert L.acdc_forward_workspace_bytes(10, 4096, 12, CX) == 0
    # invalid combinations report 0
    assert L.acdc_backward_workspace_bytes(8, 100, 2, 0, 1) == 0
    assert L.acdc_saved_bytes(-1, 64, 2, 0) == 0


class FakePtr:
    """Aligned, non-null host addresses: the validation path never
    dereferences them, and every case below fails validation before any HIP
    call."""

    def __init__(self):
        self.buf = ctypes.create_string_buffer(1024 + 64)
        base = ctypes.addressof(self.buf)
        self.base = (base + 15) & ~15

    def __call__(self, i):
        return self.base + 64 * i


def test_forward_rejects_bad_arguments(L):
    p = FakePtr()
    x, y, A, D, perm, ws = (p(i) for i in range(6))

    def fwd(x=x, y=y, A=A, D=D, perm=perm, B=4, N=64, K=2, flags=0, saved=None, sb=0, ws=ws, wsb=1 << 20):
        return L.acdc_forward(x, y, A, D, perm, B, N, K, flags, saved, sb, ws, wsb, None)

    assert fwd(N=100) == EUNSUP
    assert fwd(flags=CX | RELU) == EUNSUP
    assert fwd(flags=16) == EINVAL
    assert fwd(K=0) == EINVAL
    assert fwd(B=-1) == EINVAL
    assert fwd(x=None) == EINVAL
    assert fwd(y=None) == EINVAL
    assert fwd(A=x + 4) == EINVAL           # misaligned
    assert fwd(y=x) == EINVAL               # aliasing
    assert fwd(flags=PERM, perm=None) == EINVAL
    assert fwd(ws=None) == EWS
    assert fwd(wsb=16) == EWS
    need = L.acdc_saved_bytes(4, 64, 2, 0)
    assert fwd(saved=p(6), sb=need - 4) == EWS   # saved buffer smaller than its layout
    assert fwd(B=0) == OK                   # empty batch: nothing to do, no HIP call


def test_backward_rejects_bad_arguments(L):
    p = FakePtr()
    x, gy, A, D, perm, gx, gA, gD, ws = (p(i) for i in range(9))

    def bwd(x=x, gy=gy, A=A, D=D, perm=perm, saved=None, sb=0, gx=gx, gA=gA, gD=gD, B=4, N=64, K=2,
            flags=0, ws=ws, wsb=1 << 30):
        return L.acdc_backward(x, gy, A, D, perm, saved, sb, gx, gA, gD, B, N, K, flags, ws, wsb, None)

    assert bwd(N=48) == EUNSUP
    assert bwd(flags=CX | RELU) == EUNSUP
    assert bwd(K=-3) == EINVAL
    assert bwd(gy=None) == EINVAL
    assert bwd(gA=None) == EINVAL
    assert bwd(gx=x) == EINVAL
    assert bwd(gA=gD) == EINVAL
    assert bwd(gD=A + 8) == EINVAL
    assert bwd(flags=PERM, perm=None) == EINVAL
    assert bwd(ws=None) == EWS
    assert bwd(wsb=64) == EWS
    need = L.acdc_saved_bytes(4, 64, 2, 0)
    assert bwd(saved=p(9), sb=need - 4) == EWS   # saved buffer smaller than its layout


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(_lib.LibraryMissing):
        _lib.lib()
