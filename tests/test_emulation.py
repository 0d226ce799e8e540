"""CPU emulation of the kernel row bodies (no GPU).

The HIP kernels' __host__ __device__ bodies, the plan tables and the
fixed-order reductions run on the CPU (one thread per GPU lane, barriers for
LDS syncs) and are compared with the fp64 oracle at the same tolerance as
the GPU parity tests.  This pins the index algebra of every plan before any
GPU run; the GPU tests then pin the compiled kernels."""

import ctypes
import os
import shutil
import sys

import numpy as np
import pytest

from oracle import acdc_oracle as O
from paper_1511_05946_amd.workloads import FLAG_ACCUMULATE, FLAG_BIAS, make_bias, make_inputs
from tests.helpers import TOL_COMPLEX, TOL_REAL, rel_err, relu_safe_rows

sys.path.insert(0, os.path.join(os.path.dirname(__file__), "emu"))


@pytest.fixture(scope="module")
def emu():
    if shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"):
        pytest.skip("hipcc not available")
    import build_emu
    L = ctypes.CDLL(build_emu.build())
    P = ctypes.c_void_p
    L.acdc_emu_forward.argtypes = [P, P, P, P, P, P, ctypes.c_longlong, ctypes.c_int, ctypes.c_int,
                                   ctypes.c_uint, P]
    L.acdc_emu_backward.argtypes = [P, P, P, P, P, P, P, P, P, P, P, ctypes.c_longlong, ctypes.c_int,
                                    ctypes.c_int, ctypes.c_uint]
    L.acdc_emu_set_backward_slots.argtypes = [ctypes.c_longlong, ctypes.c_int]
    L.acdc_emu_set_backward_slots.restype = ctypes.c_int
    return L


def _p(a):
    return None if a is None else a.ctypes.data


def check(L, N, K, B, flags, seed=0, with_saved=False, perm0=False):
    x, A, D, perm, gy = make_inputs(N, K, B, flags, seed)
    if perm0:
        # the workloads keep perm[0] the identity; any permutation is valid
        perm[0] = np.random.default_rng(seed + 99).permutation(N).astype(np.int32)
    bias = make_bias(N, K, seed) if flags & FLAG_BIAS else None
    tol = TOL_COMPLEX if flags & O.FLAG_COMPLEX else TOL_REAL
    y = np.zeros_like(x)
    first = 0 if flags & O.FLAG_PERM else 1             # u_0 is stashed too with PERM
    saved = np.zeros((K - first, B, N), x.dtype) if with_saved else None
    assert L.acdc_emu_forward(_p(x), _p(y), _p(A), _p(D), _p(bias), _p(perm), B, N, K, flags, _p(saved)) == 0
    yr, cache = O.forward(x, A, D, perm, flags & 7, keep=True, B=bias)
    assert rel_err(y, yr) < tol
    if with_saved:
        # u_k in slot k - 1; with PERM u_0 (x gathered through perm[0]) in slot K - 1
        for k in range(first, K):
            assert rel_err(saved[k - 1 if k > 0 else K - 1], cache["u"][k]) < tol
    keep = relu_safe_rows(cache["v"], K) if flags & O.FLAG_RELU else np.ones(B, bool)
    x, gy = np.ascontiguousarray(x[keep]), np.ascontiguousarray(gy[keep])
    Bk = x.shape[0]
    gx, gA, gD = np.zeros_like(x), np.zeros_like(A), np.zeros_like(D)
    gB = np.zeros_like(A) if bias is not None else None
    sv = np.ascontiguousarray(saved[:, keep]) if (with_saved and K - first > 0) else None
    assert L.acdc_emu_backward(_p(x), _p(gy), _p(A), _p(D), _p(bias), _p(perm), _p(sv), _p(gx), _p(gA), _p(gD),
                               _p(gB), Bk, N, K, flags) == 0
    ref = O.backward(x, gy, A, D, perm, flags & 7, B=bias)
    assert rel_err(gx, ref[0]) < tol
    assert rel_err(gA, ref[1]) < tol
    assert rel_err(gD, ref[2]) < tol
    if bias is not None:
        assert rel_err(gB, ref[3]) < tol


@pytest.mark.parametrize("N", [8, 16, 32, 64, 128, 256, 512, 1024])
@pytest.mark.parametrize("flags", [0, O.FLAG_PERM | O.FLAG_RELU])
def test_real_small(emu, N, flags):
    check(emu, N, 3, 9, flags, seed=N)


@pytest.mark.parametrize("N", [8, 16, 64, 256, 1024])
def test_complex_small(emu, N):
    check(emu, N, 2, 5, O.FLAG_COMPLEX | O.FLAG_PERM, seed=N)


@pytest.mark.parametrize("flags", [O.FLAG_COMPLEX, O.FLAG_COMPLEX | O.FLAG_PERM])
def test_complex_4096_loads_ahead(emu, flags):
    # N = 4096 rows (adjacent pairs, 128 threads) load a and d ahead of use
    # in the forward, with and without the gather
    check(emu, 4096, 1, 1, flags, seed=41)


@pytest.mark.parametrize("flags", [O.FLAG_PERM | O.FLAG_RELU, O.FLAG_COMPLEX | O.FLAG_PERM])
@pytest.mark.parametrize("K", [1, 3])
def test_first_layer_permutation(emu, flags, K):
    check(emu, 256, K, 5, flags, seed=21 + K, perm0=True)
    check(emu, 256, K, 5, flags, seed=31 + K, perm0=True, with_saved=True)


def test_real_4096_with_saved(emu):
    check(emu, 4096, 3, 3, O.FLAG_PERM | O.FLAG_RELU, seed=1, with_saved=True)


def test_real_9216_three_waves_per_row(emu):
    check(emu, 9216, 2, 2, O.FLAG_PERM | O.FLAG_RELU, seed=2)


# Rows of 512 threads take minutes in the emulation (one OS thread per GPU
# thread, 512-way barriers); run with ACDC_EMU_WIDE=1.  The GPU parity tests
# cover these widths on every run.
wide = pytest.mark.skipif(os.environ.get("ACDC_EMU_WIDE") != "1", reason="set ACDC_EMU_WIDE=1 (slow)")


@wide
def test_real_32768_eight_waves_per_row(emu):
    check(emu, 32768, 2, 1, O.FLAG_PERM | O.FLAG_RELU | FLAG_BIAS, seed=4)


@wide
def test_complex_16384_eight_waves_per_row(emu):
    check(emu, 16384, 2, 1, O.FLAG_COMPLEX | O.FLAG_PERM, seed=5)


@pytest.mark.parametrize("N", [8, 16, 64, 256, 1024])
def test_real_bias(emu, N):
    check(emu, N, 3, 9, O.FLAG_PERM | O.FLAG_RELU | FLAG_BIAS, seed=N + 1)


def test_real_bias_4096_with_saved(emu):
    check(emu, 4096, 2, 3, O.FLAG_PERM | O.FLAG_RELU | FLAG_BIAS, seed=3, with_saved=True)


def test_accumulate_adds_to_gradients(emu):
    # ACCUMULATE adds the batch sums to what grad_A, grad_D, grad_bias hold.
    N, K, B = 64, 2, 5
    flags = O.FLAG_PERM | FLAG_BIAS
    x, A, D, perm, gy = make_inputs(N, K, B, flags, 7)
    bias = make_bias(N, K, 7)
    outs = []
    for acc in (0, FLAG_ACCUMULATE):
        gx = np.zeros_like(x)
        g = [np.full_like(A, 0.5) for _ in range(3)]
        assert emu.acdc_emu_backward(_p(x), _p(gy), _p(A), _p(D), _p(bias), _p(perm), None, _p(gx), _p(g[0]),
                                     _p(g[1]), _p(g[2]), B, N, K, flags | acc) == 0
        outs.append(g)
    for plain, added in zip(*outs):
        np.testing.assert_allclose(added, plain + 0.5, rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("n4,ntiles", [(37, t) for t in (1, 5, 24, 25, 32, 33, 61, 256)]
                         + [(16384, t) for t in (1, 12, 13, 16, 29)])
def test_reduction_order_and_value(emu, n4, ntiles):
    # The batch reduction of the parameter-gradient partials: bit for bit the
    # documented order (tiles split into P phases by t mod P, each summed in
    # increasing t, phase sums added in phase order; P = 8 below 16384 float4
    # entries, else 4), whichever branch of the grouped loads runs (groups of
    # four: phase 0 from 3P + 1 tiles on, every phase from 4P), and within
    # fp32 rounding of the exact fp64 sum.
    emu.acdc_emu_reduce4.argtypes = [ctypes.c_void_p, ctypes.c_longlong, ctypes.c_longlong, ctypes.c_void_p]
    emu.acdc_emu_reduce4.restype = ctypes.c_int
    rng = np.random.default_rng(ntiles + n4)
    part = rng.standard_normal((ntiles, n4 * 4)).astype(np.float32)
    out = np.zeros(n4 * 4, np.float32)
    P = emu.acdc_emu_reduce4(part.ctypes.data, ntiles, n4, out.ctypes.data)
    assert P == (8 if n4 < 16384 else 4)
    phases = []
    for g in range(P):
        s = np.zeros(n4 * 4, np.float32)
        for t in range(g, ntiles, P):
            s = (s + part[t]).astype(np.float32)
        phases.append(s)
    want = phases[0]
    for g in range(1, P):
        want = (want + phases[g]).astype(np.float32)
    assert np.array_equal(out, want)
    exact = part.astype(np.float64).sum(axis=0)
    assert np.max(np.abs(out - exact)) <= 1e-6 * ntiles * np.max(np.abs(part)) + 1e-7


def test_backward_over_many_tiles(emu):
    # 61 backward tiles (N = 4096: 8 rows per tile) through the emulated
    # kernels and their reduction, against the oracle
    check(emu, 4096, 1, 61 * 8, 0, seed=61)


@pytest.mark.parametrize("N,B,slots", [(1024, 83, 3), (9216, 7, 2)])
def test_persistent_workgroups_accumulate(emu, N, B, slots):
    # Persistent backward workgroups run several tiles each and add them into
    # one partial slot, fetching the slot's earlier values into LDS before
    # each sum.  With fewer slots than tiles (ragged last tile included),
    # grad_x is bitwise that of one workgroup per tile and every gradient
    # matches the oracle.
    K, flags = 3 if N == 1024 else 2, O.FLAG_PERM
    x, A, D, perm, gy = make_inputs(N, K, B, flags, 40 + slots)
    runs = []
    for s in (0, slots):
        assert emu.acdc_emu_set_backward_slots(s, N) == 1
        g = [np.zeros_like(x), np.zeros_like(A), np.zeros_like(D)]
        try:
            assert emu.acdc_emu_backward(_p(x), _p(gy), _p(A), _p(D), None, _p(perm), None, _p(g[0]), _p(g[1]),
                                         _p(g[2]), None, B, N, K, flags) == 0
        finally:
            emu.acdc_emu_set_backward_slots(0, N)
        runs.append(g)
    np.testing.assert_array_equal(runs[1][0], runs[0][0])
    ref = O.backward(x, gy, A, D, perm, flags)
    for got, want in zip(runs[1], ref):
        assert rel_err(got, want) < TOL_REAL
    # the sums really were split over slots (tiles w, w + slots, ...: not the
    # reduction's own tile phases): same values, another rounding order
    assert not np.array_equal(runs[1][1], runs[0][1])
