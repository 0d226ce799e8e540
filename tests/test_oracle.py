"""Pins for the CPU oracle (no GPU).

Each test checks the oracle against something other than itself: a library
special case (scipy's orthonormal DCT-II, numpy's FFT), a closed form of the
layer, a brute-force dense product built from the library transforms, finite
differences, or torch autograd over an independently built graph.  The last
group plants plausible mistakes in the oracle and checks that some pin fails.
"""

import json
import os

import numpy as np
import pytest
import scipy.fft

from oracle import acdc_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
P, R, CX = O.FLAG_PERM, O.FLAG_RELU, O.FLAG_COMPLEX


def rand_case(rng, B, N, K, flags, relu_input=False):
    cplx = bool(flags & CX)
    if cplx:
        x = rng.standard_normal((B, N)) + 1j * rng.standard_normal((B, N))
        A = rng.normal(1, .1, (K, N)) + 1j * rng.normal(0, .1, (K, N))
        D = rng.normal(1, .1, (K, N)) + 1j * rng.normal(0, .1, (K, N))
        gy = rng.standard_normal((B, N)) + 1j * rng.standard_normal((B, N))
    else:
        x = rng.standard_normal((B, N))
        if relu_input:
            x = np.maximum(x, 0)
        A = rng.normal(1, .1, (K, N))
        D = rng.normal(1, .1, (K, N))
        gy = rng.standard_normal((B, N))
    perm = np.stack([rng.permutation(N) for _ in range(K)])
    return x, A, D, perm, gy


def lib_forward(x, A, D, perm, flags, B=None):
    """The cascade written with library transforms only (scipy DCT-II/III
    'ortho', numpy FFT): the special case the oracle must reduce to."""
    z = np.asarray(x)
    K = A.shape[0]
    Bz = np.zeros(A.shape) if B is None else B
    for k in range(K):
        u = z[:, perm[k]] if flags & P else z
        if flags & CX:
            v = np.fft.ifft(np.fft.fft(u * A[k], axis=1) * D[k] + Bz[k], axis=1)
        else:
            v = scipy.fft.idct(scipy.fft.dct(u * A[k], type=2, norm="ortho", axis=1) * D[k] + Bz[k],
                               type=2, norm="ortho", axis=1)
        z = np.maximum(v, 0) if (flags & R and k < K - 1) else v
    return z


# ---------------------------------------------------------------- the DCT matrix

@pytest.mark.parametrize("N", [1, 2, 3, 5, 8, 16, 64, 100, 256, 1024])
def test_dct_is_scipy_orthonormal_dct2(N):
    rng = np.random.default_rng(N)
    x = rng.standard_normal((7, N))
    C = O.dct_matrix(N)
    np.testing.assert_allclose(x @ C, scipy.fft.dct(x, type=2, norm="ortho", axis=1),
                               rtol=0, atol=1e-12 * np.sqrt(N))


@pytest.mark.parametrize("N", [2, 8, 48, 256, 1024])
def test_dct_orthonormal_and_inverse(N):
    C = O.dct_matrix(N)
    np.testing.assert_allclose(C.T @ C, np.eye(N), atol=1e-12)
    np.testing.assert_allclose(C @ C.T, np.eye(N), atol=1e-12)
    x = np.random.default_rng(1).standard_normal((3, N))
    np.testing.assert_allclose(np.linalg.norm(x @ C, axis=1), np.linalg.norm(x, axis=1), rtol=1e-12)


@pytest.mark.parametrize("N", [4, 9, 64])
def test_dct_of_constant_is_dc_only(N):
    # 1 @ C = sqrt(N) e_0 for the orthonormal DCT-II.
    e0 = np.zeros(N)
    e0[0] = np.sqrt(N)
    np.testing.assert_allclose(np.ones(N) @ O.dct_matrix(N), e0, atol=1e-12)


def test_dct_small_closed_form_values():
    # N = 2: C = [[1/sqrt2, 1/sqrt2], [1/sqrt2, -1/sqrt2]] (cos(pi/4), cos(3pi/4)).
    s = 1 / np.sqrt(2)
    np.testing.assert_allclose(O.dct_matrix(2), [[s, s], [s, -s]], atol=1e-15)


@pytest.mark.parametrize("N", [1, 4, 7, 32])
def test_dft_matrix_is_numpy_fft(N):
    rng = np.random.default_rng(N)
    x = rng.standard_normal((3, N)) + 1j * rng.standard_normal((3, N))
    np.testing.assert_allclose(x @ O.dft_matrix(N), np.fft.fft(x, axis=1), atol=1e-11 * N)


# ---------------------------------------------------------- closed forms (Sec. 4)

def test_identity_layer():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 32))
    y = O.forward(x, np.ones((3, 32)), np.ones((3, 32)))
    np.testing.assert_allclose(y, x, atol=1e-12)


def test_constant_D_scales_by_A():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, 24))
    a = rng.normal(1, .1, (1, 24))
    y = O.forward(x, a, np.full((1, 24), 2.5))
    np.testing.assert_allclose(y, 2.5 * x * a, atol=1e-12)


def test_dc_only_D_gives_row_mean():
    # D = e_0: h3 keeps only the DC coefficient, so every output is mean(x * a).
    rng = np.random.default_rng(4)
    x = rng.standard_normal((6, 20))
    a = rng.normal(1, .1, (1, 20))
    d = np.zeros((1, 20))
    d[0, 0] = 1.0
    y = O.forward(x, a, d)
    np.testing.assert_allclose(y, np.repeat((x * a).mean(1, keepdims=True), 20, 1), atol=1e-12)


def test_identity_perm_equals_no_perm():
    rng = np.random.default_rng(5)
    x, A, D, _, _ = rand_case(rng, 4, 16, 3, 0)
    ident = np.tile(np.arange(16), (3, 1))
    np.testing.assert_array_equal(O.forward(x, A, D, ident, P | R), O.forward(x, A, D, None, R))


@pytest.mark.parametrize("flags", [0, P, R, P | R, CX, CX | P])
@pytest.mark.parametrize("N,K", [(8, 1), (16, 3), (48, 4), (64, 2), (256, 5)])
def test_forward_equals_library_transforms(flags, N, K):
    rng = np.random.default_rng(N * 31 + K)
    x, A, D, perm, _ = rand_case(rng, 9, N, K, flags, relu_input=bool(flags & R))
    np.testing.assert_allclose(O.forward(x, A, D, perm, flags), lib_forward(x, A, D, perm, flags),
                               atol=1e-11, rtol=1e-11)


# -------------------------------------------------- brute-force dense products

def lib_dense(A, D, perm, flags):
    """W built column by column from the library transforms, with explicit
    Python loops for the permutation and diagonal products."""
    K, N = A.shape
    cplx = bool(flags & CX)
    W = np.eye(N, dtype=complex if cplx else float)
    for k in range(K):
        if flags & P:
            Pm = np.zeros((N, N))
            for n in range(N):
                Pm[perm[k][n], n] = 1.0  # u[n] = z[perm[n]]  <=>  u = z @ Pm
            W = W @ Pm
        L = np.zeros((N, N), dtype=W.dtype)
        for i in range(N):
            e = np.zeros(N, dtype=W.dtype)
            e[i] = 1.0
            L[i] = lib_forward(e[None, :], A[k:k + 1], D[k:k + 1], None, flags & CX)[0]
        W = W @ L
    return W


@pytest.mark.parametrize("flags", [0, P, CX, CX | P])
@pytest.mark.parametrize("N,K", [(4, 1), (6, 2), (16, 3), (64, 4)])
def test_dense_operator_bruteforce(flags, N, K):
    rng = np.random.default_rng(7 + N + K)
    x, A, D, perm, _ = rand_case(rng, 5, N, K, flags)
    W = O.dense_operator(A, D, perm, flags)
    np.testing.assert_allclose(W, lib_dense(A, D, perm, flags), atol=1e-11)
    np.testing.assert_allclose(x @ W, O.forward(x, A, D, perm, flags), atol=1e-11)


def test_cascade_order_first_layer_acts_first():
    # y = x L_0 L_1: swapping the layers must change the result.
    rng = np.random.default_rng(8)
    x, A, D, perm, _ = rand_case(rng, 3, 16, 2, 0)
    y = O.forward(x, A, D)
    L0, L1 = O.layer_matrix(A[0], D[0]), O.layer_matrix(A[1], D[1])
    np.testing.assert_allclose(y, x @ L0 @ L1, atol=1e-12)
    assert np.abs(y - x @ L1 @ L0).max() > 1e-3


def test_dct_orientation_matters():
    # C D C^T != C^T D C: the reading h2 = h1 C is observable.
    rng = np.random.default_rng(9)
    C = O.dct_matrix(16)
    d = rng.normal(1, .3, 16)
    assert np.abs(C @ np.diag(d) @ C.T - C.T @ np.diag(d) @ C).max() > 1e-2


def test_layer_invariant_to_column_scaling_of_C():
    # Reading of the garbled eps_k range: any per-frequency rescaling S of C with
    # the exact inverse leaves y unchanged, so it cannot affect outputs.
    rng = np.random.default_rng(10)
    C = O.dct_matrix(12)
    S = np.diag(rng.uniform(.5, 2, 12))
    Cs = C @ S
    a, d = rng.normal(1, .1, 12), rng.normal(1, .1, 12)
    np.testing.assert_allclose(np.diag(a) @ Cs @ np.diag(d) @ np.linalg.inv(Cs),
                               O.layer_matrix(a, d), atol=1e-12)


# ------------------------------------------------------ AFDF closed forms (Sec. 3)

def test_afdf_single_layer_is_circular_convolution():
    # Remark in Sec. 3: F^{-1} diag F is circulant; x A F D F^{-1} = (x a) (*) ifft(d).
    rng = np.random.default_rng(11)
    N = 12
    x, A, D, _, _ = rand_case(rng, 3, N, 1, CX)
    c = np.fft.ifft(D[0])
    h = x * A[0]
    ref = np.zeros_like(h)
    for n in range(N):
        for m in range(N):
            ref[:, n] += h[:, m] * c[(n - m) % N]
    np.testing.assert_allclose(O.forward(x, A, D, None, CX), ref, atol=1e-12)


def test_afdf_optical_presentation():
    # Sec. 3 optical presentation: y F = (x A_1 F) D_1 R_2 D_2 ... R_K D_K with
    # R_k = F^{-1} A_k F.
    rng = np.random.default_rng(12)
    N, K = 10, 3
    x, A, D, _, _ = rand_case(rng, 2, N, K, CX)
    F = np.fft.fft(np.eye(N), axis=1)
    Finv = np.linalg.inv(F)
    M = np.diag(D[0])
    for k in range(1, K):
        M = M @ (Finv @ np.diag(A[k]) @ F) @ np.diag(D[k])
    lhs = O.forward(x, A, D, None, CX) @ F
    np.testing.assert_allclose(lhs, (x * A[0]) @ F @ M, atol=1e-10)


# ------------------------------------------------------------------- backward

def fd_grads(x, A, D, perm, flags, gy, eps=1e-6):
    def loss(x_, A_, D_):
        return float(np.sum(gy * O.forward(x_, A_, D_, perm, flags)))

    out = []
    for arr_id in range(3):
        arrs = [x.copy(), A.copy(), D.copy()]
        g = np.zeros_like(arrs[arr_id])
        for idx in np.ndindex(*g.shape):
            p = [a.copy() for a in arrs]
            m = [a.copy() for a in arrs]
            p[arr_id][idx] += eps
            m[arr_id][idx] -= eps
            g[idx] = (loss(*p) - loss(*m)) / (2 * eps)
        out.append(g)
    return out


@pytest.mark.parametrize("flags", [0, P, R, P | R])
@pytest.mark.parametrize("N,K", [(4, 1), (8, 2), (16, 3)])
def test_backward_finite_differences(flags, N, K):
    rng = np.random.default_rng(100 + N * 3 + K + flags)
    x, A, D, perm, gy = rand_case(rng, 3, N, K, flags)
    if flags & R:
        _, cache = O.forward(x, A, D, perm, flags, keep=True)
        margin = min(np.abs(cache["v"][k]).min() for k in range(K - 1)) if K > 1 else 1.0
        assert margin > 1e-4, "re-seed: ReLU kink too close for finite differences"
    gx, gA, gD = O.backward(x, gy, A, D, perm, flags)
    fx, fA, fD = fd_grads(x, A, D, perm, flags, gy)
    for a, b in ((gx, fx), (gA, fA), (gD, fD)):
        np.testing.assert_allclose(a, b, atol=1e-7, rtol=1e-6)


def _torch_graph(xt, At, Dt, perm, flags, Ct=None):
    import torch
    z = xt
    K = At.shape[0]
    for k in range(K):
        u = z[:, torch.as_tensor(perm[k])] if flags & P else z
        h1 = u * At[k]
        if flags & CX:
            v = torch.fft.ifft(torch.fft.fft(h1, dim=1) * Dt[k], dim=1)
        else:
            v = ((h1 @ Ct) * Dt[k]) @ Ct.T
        z = torch.relu(v) if (flags & R and k < K - 1) else v
    return z


@pytest.mark.parametrize("flags", [0, P, R, P | R, CX, CX | P])
def test_backward_matches_torch_autograd(flags):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(200 + flags)
    N, K, B = 32, 4, 6
    x, A, D, perm, gy = rand_case(rng, B, N, K, flags)
    dt = torch.complex128 if flags & CX else torch.float64
    xt = torch.tensor(x, dtype=dt, requires_grad=True)
    At = torch.tensor(A, dtype=dt, requires_grad=True)
    Dt = torch.tensor(D, dtype=dt, requires_grad=True)
    Ct = torch.tensor(scipy.fft.dct(np.eye(N), type=2, norm="ortho", axis=1), dtype=torch.float64)
    y = _torch_graph(xt, At, Dt, perm, flags, Ct)
    y.backward(torch.tensor(gy, dtype=dt))
    gx, gA, gD = O.backward(x, gy, A, D, perm, flags)
    np.testing.assert_allclose(gx, xt.grad.numpy(), atol=1e-11)
    np.testing.assert_allclose(gA, At.grad.numpy(), atol=1e-10)
    np.testing.assert_allclose(gD, Dt.grad.numpy(), atol=1e-10)


def test_backward_batch_split_additivity():
    rng = np.random.default_rng(300)
    x, A, D, perm, gy = rand_case(rng, 10, 16, 3, P | R)
    gx, gA, gD = O.backward(x, gy, A, D, perm, P | R)
    gx1, gA1, gD1 = O.backward(x[:4], gy[:4], A, D, perm, P | R)
    gx2, gA2, gD2 = O.backward(x[4:], gy[4:], A, D, perm, P | R)
    np.testing.assert_allclose(gx, np.concatenate([gx1, gx2]), atol=1e-13)
    np.testing.assert_allclose(gA, gA1 + gA2, atol=1e-12)
    np.testing.assert_allclose(gD, gD1 + gD2, atol=1e-12)


# --------------------------------- wide rows: library transforms for dense ones

@pytest.mark.parametrize("flags", [P | R, CX | P])
@pytest.mark.parametrize("N", [64, 1024])
def test_library_transform_path_equals_dense(monkeypatch, flags, N):
    # Rows wider than DENSE_MAX apply C, C^T (F, F^{-1}) through scipy/numpy
    # transforms; on widths where both exist the two paths agree.
    rng = np.random.default_rng(600 + N + flags)
    x, A, D, perm, gy = rand_case(rng, 5, N, 3, flags, relu_input=True)
    b = rand_bias(rng, 3, N, bool(flags & CX))
    dense = O.forward(x, A, D, perm, flags, B=b), O.backward(x, gy, A, D, perm, flags, B=b)
    monkeypatch.setattr(O, "DENSE_MAX_REAL", 4)
    monkeypatch.setattr(O, "DENSE_MAX_COMPLEX", 4)
    lib = O.forward(x, A, D, perm, flags, B=b), O.backward(x, gy, A, D, perm, flags, B=b)
    np.testing.assert_allclose(lib[0], dense[0], atol=1e-11)
    for a, c in zip(lib[1], dense[1]):
        np.testing.assert_allclose(a, c, atol=1e-10)


def test_dense_path_serves_the_mixed_radix_width():
    # N = 9216 = 2^10 * 3^2 (the Sec. 6.2 feature width) runs on the dense
    # Sec. 4 matrix, which must agree with scipy's orthonormal DCT-II there
    # too: a wrong angle reduction or index would show at this width first.
    N = 9216
    assert N <= O.dense_limit(False)
    rng = np.random.default_rng(9216)
    x = rng.standard_normal((3, N))
    C = O.dct_matrix(N)
    np.testing.assert_allclose(x @ C, scipy.fft.dct(x, type=2, norm="ortho", axis=1), rtol=0, atol=1e-11)
    np.testing.assert_allclose(x @ C @ C.T, x, rtol=0, atol=1e-11)
    # and a two-layer permuted ReLU cascade: dense oracle vs library transforms
    x, A, D, perm, gy = rand_case(rng, 3, N, 2, P | R, relu_input=True)
    np.testing.assert_allclose(O.forward(x, A, D, perm, P | R), lib_forward(x, A, D, perm, P | R),
                               rtol=0, atol=1e-10)


# ------------------------------------- ReLU decisions taken as an input

@pytest.mark.parametrize("flags", [R, P | R])
def test_own_decisions_reproduce_default(flags):
    # Passing the oracle's own decisions changes nothing, bit for bit.
    rng = np.random.default_rng(700 + flags)
    x, A, D, perm, gy = rand_case(rng, 9, 32, 4, flags, relu_input=True)
    b = rand_bias(rng, 4, 32, False)
    y, c = O.forward(x, A, D, perm, flags, keep=True, B=b)
    m = O.relu_decisions(c, 4)
    assert m.shape == (3, 9, 32) and m.dtype == bool
    assert np.array_equal(O.forward(x, A, D, perm, flags, B=b, masks=m), y)
    for u, v in zip(O.backward(x, gy, A, D, perm, flags, B=b),
                    O.backward(x, gy, A, D, perm, flags, B=b, masks=m)):
        assert np.array_equal(u, v)
    assert O.mask_disagreements(m, c, 4, 1e-4) == 0


def test_given_decisions_are_used_consistently():
    # With decisions fixed (here: random, not the oracle's), the cascade is
    # linear in x, a and d separately, so the analytic backward must match
    # finite differences of the forward under the same decisions.  This pins
    # that forward and backward apply the given masks at the same places.
    rng = np.random.default_rng(710)
    N, K, flags = 8, 3, P | R
    x, A, D, perm, gy = rand_case(rng, 2, N, K, flags)
    m = rng.random((K - 1, 2, N)) < 0.5

    def loss(x_, A_, D_):
        return float(np.sum(gy * O.forward(x_, A_, D_, perm, flags, masks=m)))

    gx, gA, gD = O.backward(x, gy, A, D, perm, flags, masks=m)
    eps = 1e-6
    for arr_id, got in enumerate((gx, gA, gD)):
        arrs = [x, A, D]
        for idx in np.ndindex(*got.shape):
            p = [a.copy() for a in arrs]
            q = [a.copy() for a in arrs]
            p[arr_id][idx] += eps
            q[arr_id][idx] -= eps
            assert abs((loss(*p) - loss(*q)) / (2 * eps) - got[idx]) < 1e-7 + 1e-6 * abs(got[idx])
    # and the decisions matter: the default ones give a different result
    assert not np.allclose(O.backward(x, gy, A, D, perm, flags)[0], gx)


def test_mask_disagreements_counts_only_clear_decisions():
    # A decision flipped where |v| is far from zero is counted; one flipped
    # inside the tie band is not.
    v = np.array([[[3.0, -2.0, 1e-9, -1e-9]]])  # one layer, one row
    cache = {"v": [v[0]]}
    rms = np.sqrt(np.mean(v[0] ** 2))
    own = v > 0
    assert O.mask_disagreements(own, cache, 2, 1e-4) == 0
    near = own.copy()
    near[0, 0, 2] = ~near[0, 0, 2]
    near[0, 0, 3] = ~near[0, 0, 3]
    assert O.mask_disagreements(near, cache, 2, 1e-4) == 0
    far = own.copy()
    far[0, 0, 1] = ~far[0, 0, 1]
    assert O.mask_disagreements(far, cache, 2, 1e-4) == 1
    assert O.mask_disagreements(far, cache, 2, 2.0 / rms + 1e-9) == 0
    with pytest.raises(ValueError):
        O.forward(np.ones((1, 4)), np.ones((2, 4)), np.ones((2, 4)), None, 0, masks=own)  # no RELU flag
    with pytest.raises(ValueError):
        O.forward(np.ones((1, 4)), np.ones((3, 4)), np.ones((3, 4)), None, R, masks=own)  # wrong K


# ------------------------------------------- D-domain bias (Sec. 6.2)

def rand_bias(rng, K, N, cplx):
    b = rng.normal(0, .3, (K, N))
    return b + 1j * rng.normal(0, .3, (K, N)) if cplx else b


@pytest.mark.parametrize("cplx", [False, True])
def test_bias_with_zero_D_is_inverse_transform_of_bias(cplx):
    # D = 0 removes the input: every output row is b C^{-1} (scipy's
    # orthonormal DCT-III) or b F^{-1} (numpy's inverse FFT).
    rng = np.random.default_rng(500 + cplx)
    flags = CX if cplx else 0
    x, A, D, perm, _ = rand_case(rng, 5, 16, 1, flags)
    b = rand_bias(rng, 1, 16, cplx)
    y = O.forward(x, A, np.zeros_like(D), perm, flags, B=b)
    ref = np.fft.ifft(b[0]) if cplx else scipy.fft.idct(b[0], type=2, norm="ortho")
    np.testing.assert_allclose(y, np.broadcast_to(ref, y.shape), atol=1e-14)


@pytest.mark.parametrize("flags", [0, P | R, CX | P])
def test_bias_forward_equals_library_transforms(flags):
    rng = np.random.default_rng(510 + flags)
    x, A, D, perm, _ = rand_case(rng, 7, 32, 3, flags, relu_input=True)
    b = rand_bias(rng, 3, 32, bool(flags & CX))
    np.testing.assert_allclose(O.forward(x, A, D, perm, flags, B=b), lib_forward(x, A, D, perm, flags, b),
                               atol=1e-12)


@pytest.mark.parametrize("cplx", [False, True])
def test_bias_gradient_single_layer_closed_form(cplx):
    # One layer: dL/db = sum_rows g C (scipy's orthonormal DCT-II of each
    # gradient row) or sum_rows g F / N (numpy FFT / N); the other gradients
    # do not depend on b.
    rng = np.random.default_rng(520 + cplx)
    flags = CX if cplx else 0
    x, A, D, perm, gy = rand_case(rng, 6, 16, 1, flags)
    b = rand_bias(rng, 1, 16, cplx)
    gx, gA, gD, gB = O.backward(x, gy, A, D, perm, flags, B=b)
    ref = (np.fft.fft(gy, axis=1) / 16 if cplx else scipy.fft.dct(gy, type=2, norm="ortho", axis=1)).sum(0)
    np.testing.assert_allclose(gB[0], ref, atol=1e-12)
    gx0, gA0, gD0 = O.backward(x, gy, A, D, perm, flags)
    for a, c in ((gx, gx0), (gA, gA0), (gD, gD0)):
        np.testing.assert_allclose(a, c, atol=1e-13)


def test_bias_gradient_finite_differences():
    rng = np.random.default_rng(530)
    flags = P | R
    x, A, D, perm, gy = rand_case(rng, 3, 8, 3, flags)
    b = rand_bias(rng, 3, 8, False)
    _, cache = O.forward(x, A, D, perm, flags, keep=True, B=b)
    assert min(np.abs(cache["v"][k]).min() for k in range(2)) > 1e-4, "re-seed: ReLU kink too close"
    gB = O.backward(x, gy, A, D, perm, flags, B=b)[3]
    eps = 1e-6
    fd = np.zeros_like(b)
    for idx in np.ndindex(*b.shape):
        bp, bm = b.copy(), b.copy()
        bp[idx] += eps
        bm[idx] -= eps
        fd[idx] = (np.sum(gy * lib_forward(x, A, D, perm, flags, bp)) -
                   np.sum(gy * lib_forward(x, A, D, perm, flags, bm))) / (2 * eps)
    np.testing.assert_allclose(gB, fd, atol=1e-7, rtol=1e-6)


@pytest.mark.parametrize("flags", [P | R, CX | P])
def test_bias_backward_matches_torch_autograd(flags):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(540 + flags)
    N, K, B = 32, 3, 5
    cplx = bool(flags & CX)
    x, A, D, perm, gy = rand_case(rng, B, N, K, flags)
    b = rand_bias(rng, K, N, cplx)
    dt = torch.complex128 if cplx else torch.float64
    Ct = torch.tensor(scipy.fft.dct(np.eye(N), type=2, norm="ortho", axis=1), dtype=torch.float64)
    xt, At, Dt, Bt = (torch.tensor(v, dtype=dt, requires_grad=True) for v in (x, A, D, b))
    z = xt
    for k in range(K):
        u = z[:, torch.as_tensor(perm[k])] if flags & P else z
        if cplx:
            v = torch.fft.ifft(torch.fft.fft(u * At[k], dim=1) * Dt[k] + Bt[k], dim=1)
        else:
            v = (((u * At[k]) @ Ct) * Dt[k] + Bt[k]) @ Ct.T
        z = torch.relu(v) if (flags & R and k < K - 1) else v
    z.backward(torch.tensor(gy, dtype=dt))
    gx, gA, gD, gB = O.backward(x, gy, A, D, perm, flags, B=b)
    for a, t in ((gx, xt), (gA, At), (gD, Dt), (gB, Bt)):
        np.testing.assert_allclose(a, t.grad.numpy(), atol=1e-10)


def test_bias_planted_mistakes_are_caught(monkeypatch):
    good = O.forward

    def spatial_bias(x, A, D, perm=None, flags=0, keep=False, B=None):
        # bias added after the inverse transform instead of in the D domain
        y = good(x, A, D, perm, flags, keep)
        if B is None:
            return y
        if keep:
            return y[0] + B[-1], y[1]
        return y + B[-1]
    monkeypatch.setattr(O, "forward", spatial_bias)
    with pytest.raises(AssertionError):
        test_bias_with_zero_D_is_inverse_transform_of_bias(False)
    monkeypatch.setattr(O, "forward", good)

    good_bwd = O.backward

    def spatial_grad(x, gy, A, D, perm=None, flags=0, B=None):
        # dL/db taken as the spatial row sum instead of its transform
        out = good_bwd(x, gy, A, D, perm, flags, B)
        if B is None:
            return out
        return out[:3] + (np.broadcast_to(np.asarray(gy).sum(0), np.shape(B)).copy(),)
    monkeypatch.setattr(O, "backward", spatial_grad)
    with pytest.raises(AssertionError):
        test_bias_gradient_single_layer_closed_form(False)
    monkeypatch.setattr(O, "backward", good_bwd)


# ------------------------------------------------------ paper's printed numbers

def test_cost_model_matches_paper_printed_numbers():
    g = json.load(open(os.path.join(GOLDEN, "paper_cost_model.json")))
    lo, hi = g["ai_range_N"]
    # printed to one decimal (9.25 appears as 9.3, so allow half a unit)
    assert abs(O.arithmetic_intensity(lo) - g["ai_range_printed"][0]) <= 0.05 + 1e-12
    assert abs(O.arithmetic_intensity(hi) - g["ai_range_printed"][1]) <= 0.05 + 1e-12
    assert round(g["titan_x_peak_gflops"] / g["titan_x_peak_gbps"]) == g["titan_x_ridge_flop_per_byte_approx"]


def test_flop_counts_against_hand_computed_values():
    # The roofline's numerator.  Values computed by hand from the Sec. 5
    # count (4N + 5 N log2 N per real row-layer) and, for AFDF rows, two
    # complex N-point FFTs in the same convention (5 N log2 N each) plus two
    # complex diagonal products (6 flops per complex multiply, N each).
    # Both the oracle's count and bench.py's own copy must reproduce them.
    import bench
    g = json.load(open(os.path.join(GOLDEN, "paper_cost_model.json")))
    for case in g["flops_per_row_layer"]:
        N, cplx, want = case["N"], case["complex"], case["flops"]
        assert O.flops_per_row_layer(N, cplx) == pytest.approx(want, rel=1e-12)
        assert bench.flops_row_layer(N, cplx) == pytest.approx(want, rel=1e-12)


# ----------------------------------------- planted mistakes must be caught (CPU)

def _pins_pass():
    """A compact subset of the pins above, run against the (possibly patched)
    oracle.  Returns False as soon as one fails."""
    rng = np.random.default_rng(400)
    try:
        for flags in (P | R, CX | P):
            x, A, D, perm, gy = rand_case(rng, 4, 8, 2, flags)
            np.testing.assert_allclose(O.forward(x, A, D, perm, flags),
                                       lib_forward(x, A, D, perm, flags), atol=1e-10)
        test_backward_matches_torch_autograd(P | R)
        test_backward_matches_torch_autograd(CX | P)
    except AssertionError:
        return False
    return True


def test_planted_mistakes_are_caught(monkeypatch):
    assert _pins_pass()
    good_dct = O.dct_matrix

    # 1) transposed DCT (C^T D C instead of C D C^T)
    monkeypatch.setattr(O, "dct_matrix", lambda N: good_dct(N).T.copy())
    assert not _pins_pass()
    monkeypatch.setattr(O, "dct_matrix", good_dct)

    # 2) wrong normalisation eps_0 = 1 (breaks orthogonality)
    def bad_eps(N):
        C = good_dct(N).copy()
        C[:, 0] *= np.sqrt(2)
        return C
    monkeypatch.setattr(O, "dct_matrix", bad_eps)
    assert not _pins_pass()
    monkeypatch.setattr(O, "dct_matrix", good_dct)

    # 3) DFT sign flipped
    good_dft = O.dft_matrix
    monkeypatch.setattr(O, "dft_matrix", lambda N: np.conj(good_dft(N)))
    assert not _pins_pass()
    monkeypatch.setattr(O, "dft_matrix", good_dft)

    # 4) scatter instead of gather for the permutation
    good_fwd = O.forward

    def scatter_fwd(x, A, D, perm=None, flags=0, keep=False):
        inv = None if perm is None else np.argsort(np.asarray(perm), axis=1)
        return good_fwd(x, A, D, inv, flags, keep)
    monkeypatch.setattr(O, "forward", scatter_fwd)
    assert not _pins_pass()
    monkeypatch.setattr(O, "forward", good_fwd)

    # 5) a dropped conjugate / sign in the backward (perturb the analytic
    #    backward by computing it on conj(D) for the complex path)
    good_bwd = O.backward

    def bad_bwd(x, gy, A, D, perm=None, flags=0):
        return good_bwd(x, gy, A, np.conj(D) if flags & CX else D, perm, flags)
    monkeypatch.setattr(O, "backward", bad_bwd)
    assert not _pins_pass()
    monkeypatch.setattr(O, "backward", good_bwd)

    assert _pins_pass()
