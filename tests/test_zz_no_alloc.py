"""The no-allocation forward (acdc_forward_noalloc) through the C ABI on the
GPU: bit for bit the result of acdc_forward (same kernels, same per-layer
coefficients), on two calls in a row, the second with a smaller batch and
fewer layers, so that it reads a scratch array still holding the first
call's contents."""

import ctypes

import numpy as np
import pytest

from paper_1511_05946_amd.workloads import FLAG_BIAS, make_bias, make_inputs

pytestmark = pytest.mark.gpu

PERM, RELU, CX = 1, 2, 4


@pytest.fixture(scope="module")
def env():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1511_05946_amd import _lib
    return torch, _lib.lib()


def _dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _nb(t):
    return 0 if t is None else t.numel() * t.element_size()


def _forward_both(torch, L, N, K, B, flags, seed):
    print(f"[case] no-alloc forward N={N} K={K} B={B} flags={flags}", flush=True)
    x, A, D, perm, _ = make_inputs(N, K, B, flags, seed)
    bias = make_bias(N, K, seed) if flags & FLAG_BIAS else None
    xt, At, Dt, pt = (_dev(torch, a) for a in (x, A, D, perm))
    bt = _dev(torch, bias) if bias is not None else None
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    nsaved = L.acdc_saved_bytes(B, N, K, flags) // xt.element_size()   # elements of x's dtype
    outs = []
    for which in ("plain", "noalloc"):
        y = torch.full_like(xt, float("nan"))
        saved = torch.full((max(nsaved, 1),), float("nan"), dtype=xt.dtype, device="cuda")
        if which == "plain":
            wsb = L.acdc_forward_workspace_size(B, N, K, flags)
            ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device="cuda")
            rc = L.acdc_forward(_p(xt), _p(y), _p(At), _p(Dt), _p(bt), _p(pt), B, N, K, flags, _p(saved),
                                _nb(saved), _p(ws), wsb, stream)
        else:
            rc = L.acdc_forward_noalloc(_p(xt), _p(y), _p(At), _p(Dt), _p(bt), _p(pt), B, N, K, flags, _p(saved),
                                        _nb(saved), stream)
        assert rc == 0, (which, rc)
        torch.cuda.synchronize()
        outs.append((y.cpu().numpy(), saved.cpu().numpy()[:nsaved]))
    (y0, s0), (y1, s1) = outs
    assert np.isfinite(y1).all()
    assert np.array_equal(y0, y1)
    assert np.array_equal(s0, s1)


@pytest.mark.parametrize("N,flags", [(4096, PERM | RELU), (1024, PERM | RELU | FLAG_BIAS), (9216, PERM | RELU),
                                     (2048, CX | PERM)])
def test_noalloc_forward_matches_forward(env, N, flags):
    torch, L = env
    assert L.acdc_prepare(N, flags) == 0
    _forward_both(torch, L, N, 12, 64, flags, seed=N + 1)
    _forward_both(torch, L, N, 3, 17, flags, seed=N + 2)      # smaller input, scratch holds the last call's data


def test_noalloc_forward_rejects_what_it_cannot_serve(env):
    torch, L = env
    assert L.acdc_prepare(4096, PERM) == 0
    x = torch.zeros(4, 4096, device="cuda")
    y = torch.zeros_like(x)
    A = torch.ones(300, 4096, device="cuda")
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    # 300 layers of 4096 need 19.7 MB of coefficients: more than the 16 MiB array
    assert L.acdc_forward_noalloc(_p(x), _p(y), _p(A), _p(A), None, None, 4, 4096, 300, 0, None, 0, s) == -3
    # the multi-pass path's workspace grows with the batch: not served
    xm = torch.zeros(2, 65536, device="cuda")
    Am = torch.ones(1, 65536, device="cuda")
    assert L.acdc_forward_noalloc(_p(xm), _p(torch.zeros_like(xm)), _p(Am), _p(Am), None, None, 2, 65536, 1, 0,
                                  None, 0, s) == -2
