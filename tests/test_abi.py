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
    for n in ("acdc_forward", "acdc_backward", "acdc_backward_workspace_size", "acdc_prepare",
              "acdc_status_string", "acdc_last_hip_error", "acdc_supported", "acdc_sync_timeouts"):
        assert n in names


def test_every_declared_symbol_is_exported(L):
    for n in declared_functions():
        assert hasattr(L, n), n
        assert n in _lib.SIGNATURES, f"binding lacks a signature for {n}"


def test_supported_widths(L):
    for N in (8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096, 8192, 9216, 16384, 32768):
        assert L.acdc_supported(N, 0) == 1
        assert L.acdc_supported(N, PERM | RELU) == 1
    for N in (8, 64, 1024, 4096, 8192, 16384):
        assert L.acdc_supported(N, CX | PERM) == 1
    for N in (0, 2, 4, 6, 12, 100, 1000, 3072, 1 << 23):
        assert L.acdc_supported(N, 0) == 0
    # multi-pass: real rows of any power of two 256 ... 2^22, complex rows
    # 256 ... 2^21 (the same FFT lengths)
    MP = 32
    for N in (65536, 1 << 19, 1 << 22):
        assert L.acdc_supported(N, PERM | RELU) == 1
    for N in (32768, 65536, 1 << 21):
        assert L.acdc_supported(N, CX | PERM) == 1
    assert L.acdc_supported(1 << 22, CX) == 0
    for N in (256, 4096, 32768):
        assert L.acdc_supported(N, MP | PERM) == 1
        assert L.acdc_supported(N, MP | CX | PERM) == 1
    for N in (128, 9216, 3072):
        assert L.acdc_supported(N, MP) == 0
        assert L.acdc_supported(N, MP | CX) == 0
    assert L.acdc_supported(65536, CX | RELU) == 0
    assert L.acdc_supported(9216, CX) == 0
    assert L.acdc_supported(4096, CX | RELU) == 0
    assert L.acdc_supported(4096, 8) == 1          # BIAS
    assert L.acdc_supported(4096, 64) == 0         # unknown flag bit


def test_status_strings(L):
    for rc in (OK, EINVAL, EUNSUP, EWS, EHIP, 99):
        assert isinstance(L.acdc_status_string(rc), bytes)
    assert L.acdc_status_string(OK) == b"ok"


def test_sizes(L):
    assert L.acdc_saved_bytes(8192, 4096, 12, PERM | RELU) == 12 * 8192 * 4096 * 4   # u_0 .. u_11
    assert L.acdc_saved_bytes(8192, 4096, 12, RELU) == 11 * 8192 * 4096 * 4          # u_1 .. u_11
    assert L.acdc_saved_bytes(10, 64, 1, 0) == 0
    assert L.acdc_saved_bytes(10, 64, 1, PERM) == 10 * 64 * 4
    assert L.acdc_saved_bytes(10, 64, 3, CX) == 2 * 10 * 64 * 8
    ws_saved = L.acdc_backward_workspace_size(8192, 4096, 12, PERM | RELU, 1)
    ws_recompute = L.acdc_backward_workspace_size(8192, 4096, 12, PERM | RELU, 0)
    assert ws_saved > 0 and ws_recompute >= ws_saved + 12 * 8192 * 4096 * 4
    assert L.acdc_forward_workspace_size(8192, 4096, 12, 0) > 0
    assert L.acdc_forward_workspace_size(10, 4096, 12, CX) == 0
    # invalid combinations report 0
    assert L.acdc_backward_workspace_size(8, 100, 2, 0, 1) == 0
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


BIAS, ACC = 8, 16


def test_forward_rejects_bad_arguments(L):
    p = FakePtr()
    x, y, A, D, perm, ws, b = (p(i) for i in range(7))

    def fwd(x=x, y=y, A=A, D=D, b=None, perm=perm, B=4, N=64, K=2, flags=0, saved=None, sb=0, ws=ws,
            wsb=1 << 20):
        return L.acdc_forward(x, y, A, D, b, perm, B, N, K, flags, saved, sb, ws, wsb, None)

    assert fwd(N=100) == EUNSUP
    assert fwd(flags=CX | RELU) == EUNSUP
    assert fwd(flags=CX | BIAS, b=b) == EUNSUP
    assert fwd(flags=64) == EINVAL
    assert fwd(K=0) == EINVAL
    assert fwd(B=-1) == EINVAL
    assert fwd(x=None) == EINVAL
    assert fwd(y=None) == EINVAL
    assert fwd(A=x + 4) == EINVAL           # misaligned
    assert fwd(y=x) == EINVAL               # aliasing
    assert fwd(y=b, b=b, flags=BIAS) == EINVAL
    assert fwd(flags=PERM, perm=None) == EINVAL
    assert fwd(flags=BIAS) == EINVAL        # bias required with BIAS
    assert fwd(flags=BIAS, b=b + 4) == EINVAL
    assert fwd(ws=None) == EWS
    assert fwd(wsb=16) == EWS
    need = L.acdc_saved_bytes(4, 64, 2, 0)
    assert fwd(saved=p(7), sb=need - 4) == EWS   # saved buffer smaller than its layout
    assert fwd(B=0) == OK                   # empty batch: nothing to do, no HIP call


def test_backward_rejects_bad_arguments(L):
    p = FakePtr()
    x, gy, A, D, perm, gx, gA, gD, ws, b, gb = (p(i) for i in range(11))

    def bwd(x=x, gy=gy, A=A, D=D, b=None, perm=perm, saved=None, sb=0, gx=gx, gA=gA, gD=gD, gb=None, B=4,
            N=64, K=2, flags=0, ws=ws, wsb=1 << 30):
        return L.acdc_backward(x, gy, A, D, b, perm, saved, sb, gx, gA, gD, gb, B, N, K, flags, ws, wsb, None)

    assert bwd(N=48) == EUNSUP
    assert bwd(flags=CX | RELU) == EUNSUP
    assert bwd(flags=CX | BIAS, b=b, gb=gb) == EUNSUP
    assert bwd(K=-3) == EINVAL
    assert bwd(gy=None) == EINVAL
    assert bwd(gA=None) == EINVAL
    assert bwd(gx=x) == EINVAL
    assert bwd(gA=gD) == EINVAL
    assert bwd(gD=A + 8) == EINVAL
    assert bwd(flags=PERM, perm=None) == EINVAL
    assert bwd(flags=BIAS, b=b) == EINVAL        # grad_bias required with BIAS
    assert bwd(flags=BIAS, gb=gb) == EINVAL      # bias required with BIAS
    assert bwd(flags=BIAS, b=b, gb=gA) == EINVAL  # aliased gradients
    assert bwd(flags=BIAS | ACC, b=b, gb=gb + 4) == EINVAL
    assert bwd(ws=None) == EWS
    assert bwd(wsb=64) == EWS
    need = L.acdc_saved_bytes(4, 64, 2, 0)
    assert bwd(saved=p(11), sb=need - 4) == EWS   # saved buffer smaller than its layout
    # the bias gradient needs workspace even for an empty batch
    assert L.acdc_backward_workspace_size(0, 64, 2, BIAS, 1) > 0
    assert bwd(B=0, flags=BIAS, b=b, gb=gb, ws=None) == EWS


def test_bias_workspace_sizes(L):
    plain = L.acdc_backward_workspace_size(8192, 4096, 12, PERM | RELU, 1)
    biased = L.acdc_backward_workspace_size(8192, 4096, 12, PERM | RELU | BIAS, 1)
    # one more N-float partial per tile and layer, plus the [K, N] batch sums
    assert biased >= plain + 12 * 4096 * 4
    assert L.acdc_supported(4096, PERM | RELU | BIAS | ACC) == 1
    assert L.acdc_supported(4096, CX | BIAS) == 0
    assert L.acdc_supported(4096, CX | ACC) == 1


def test_multipass_workspace_sizes(L):
    MP = 32
    B, N, K = 64, 65536, 4
    rows_real, rows_cx = B * N * 4, B * N * 8  # bytes of one batch of rows
    # forward: spectra and layer buffer, plus the permuted input with PERM
    assert L.acdc_forward_workspace_size(B, N, K, PERM) >= 3 * rows_real
    assert L.acdc_forward_workspace_size(B, N, K, CX | PERM) >= 3 * rows_cx
    assert L.acdc_forward_workspace_size(B, N, K, CX) < L.acdc_forward_workspace_size(B, N, K, CX | PERM)
    # backward: the h and g spectra (one batch each), dL/dv, the next g, the
    # dL/da image (+ dL/du before the complex adjoint permutation), and the
    # recompute stash when nothing is saved
    assert L.acdc_backward_workspace_size(B, N, K, PERM, 1) >= 5 * rows_real
    assert L.acdc_backward_workspace_size(B, N, K, CX | PERM, 1) >= 6 * rows_cx
    saved = L.acdc_saved_bytes(B, N, K, CX | PERM)
    assert saved == K * rows_cx
    assert (L.acdc_backward_workspace_size(B, N, K, CX | PERM, 0)
            >= L.acdc_backward_workspace_size(B, N, K, CX | PERM, 1) + saved)
    # forcing the multi-pass path at a fused width needs more workspace
    assert L.acdc_forward_workspace_size(B, 4096, K, CX | PERM | MP) > L.acdc_forward_workspace_size(B, 4096, K, CX | PERM)
    # unsupported: complex rows past 2^21
    assert L.acdc_forward_workspace_size(B, 1 << 22, K, CX) == 0


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(_lib.LibraryMissing):
        _lib.lib()


def test_binding_checks_shapes_before_any_library_call(L):
    # The library takes raw pointers: a tensor of the wrong shape must be
    # rejected by the binding (ValueError) before it reaches acdc_forward /
    # acdc_backward.  CPU tensors suffice, since shapes are checked first.
    torch = pytest.importorskip("torch")
    import paper_1511_05946_amd.acdc as acdc
    B, N, K = 3, 64, 2
    x = torch.zeros(B, N)
    A = torch.ones(K, N)
    perm = torch.arange(N, dtype=torch.int32).repeat(K, 1)
    bad = {
        "A width": dict(A=torch.ones(K, N + 4)),
        "D": dict(D=torch.ones(K + 1, N)),
        "perm": dict(perm=torch.arange(N - 4, dtype=torch.int32).repeat(K, 1)),
        "bias": dict(bias=torch.zeros(K, N - 4)),
        "out": dict(out=torch.zeros(B + 1, N)),
        "saved": dict(saved=torch.zeros(5)),
    }
    for what, kw in bad.items():
        args = dict(x=x, A=A, D=A.clone(), perm=perm, flags=PERM)
        args.update(kw)
        with pytest.raises(ValueError):
            acdc.forward(**args)
    gbad = {
        "grad_y": dict(grad_y=torch.zeros(B, N + 4)),
        "grad_x": dict(out=torch.zeros(B - 1, N)),
        "grad_A": dict(grads=(torch.zeros(K, N - 4), torch.zeros(K, N))),
        "grad_D": dict(grads=(torch.zeros(K, N), torch.zeros(K - 1, N))),
        "grads arity": dict(grads=(torch.zeros(K, N),)),
        "grad_bias": dict(bias=torch.zeros(K, N), grads=(torch.zeros(K, N), torch.zeros(K, N), torch.zeros(K, 1))),
        "perm": dict(perm=torch.zeros(K, N + 4, dtype=torch.int32)),
    }
    for what, kw in gbad.items():
        args = dict(x=x, grad_y=torch.zeros(B, N), A=A, D=A.clone(), perm=perm, flags=PERM)
        args.update(kw)
        with pytest.raises(ValueError):
            acdc.backward(**args)


def test_noalloc_forward_rejects_on_the_host(L):
    # acdc_forward_noalloc refuses, before any HIP call, what its fixed
    # scratch array cannot hold (more than 2^20 layer-elements of real rows)
    # and the multi-pass path (workspace grows with the batch)
    P = ctypes.c_void_p
    x = P(0x1000)
    y = P(0x2000)
    A = P(0x3000)
    D = P(0x4000)
    assert L.acdc_forward_noalloc(x, y, A, D, None, None, 4, 4096, 300, 0, None, 0, None) == EWS
    assert L.acdc_forward_noalloc(x, y, A, D, None, None, 4, 65536, 1, 0, None, 0, None) == EUNSUP
    assert L.acdc_forward_noalloc(x, y, A, D, None, None, 4, 4096, 1, 1 << 20, None, 0, None) == EINVAL
    assert L.acdc_status_string(-5).decode().startswith("width not prepared")
