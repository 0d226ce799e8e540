"""Plain CPU oracle for deep ACDC / AFDF cascades.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  The product path
(the HIP library and its Python binding) never calls it, and it shares no code,
tables or constants with that path.

Everything is computed in float64 (complex128 for the AFDF variant) with dense
O(N^2) matrices built directly from their definitions (real rows up to
N = DENSE_MAX_REAL = 16384, complex rows up to DENSE_MAX_COMPLEX = 8192;
wider rows apply the same matrices through scipy's / numpy's transforms,
which the pins equate with the dense matrices).  There is no blocking and no
fusion: each function follows the paper's statement of the layer in the
order the paper gives it.

Paper: Moczulski, Denil, Appleyard, de Freitas, "ACDC: A Structured Efficient
Linear Layer", ICLR 2016 (arXiv:1511.05946).

Conventions (row vectors throughout, as in the paper's Sec. 1 eq. (1) y = xW):

* ``x``            [B, N] layer-cascade input
* ``A``, ``D``     [K, N] diagonals a_k, d_k of layer k (A_k = diag(a_k))
* ``perm``         [K, N] int; ``perm[k]`` *gathers* the input of layer k:
                   u_k[n] = z_{k-1}[perm[k][n]]
* ``B``            [K, N] optional additive bias of each layer's D-domain
                   term, h3 = h2 * d_k + b_k (Sec. 6.2: biases added to the
                   D matrices, none on A)
* ``flags``        bit 0 PERM, bit 1 RELU (after layers 0..K-2), bit 2 COMPLEX

Readings of the paper used here:

* DCT index range: n, k in [0, N) and eps_0 = 1/sqrt(2) only (Sec. 4, the
  c_nk definition; the "k = N" clause is a DCT-I leftover -- only this reading
  makes the matrix orthogonal, which Sec. 4 states).
* Orientation: n is the spatial index, so ``h2 = h1 @ C`` is the DCT-II and
  ``@ C.T`` (= C^{-1}) the DCT-III (Sec. 4 derivative block: h2 = h1 C).
* Batch reduction of dL/da, dL/dd: sum over rows (Sec. 4 gives per-example
  derivatives).
* ReLU derivative at 0 is 0 (strict v > 0).
* ReLU decisions may be given as an input (``masks``): where a pre-ReLU value
  lies within rounding of zero, an fp32 evaluation of the same cascade may
  legitimately decide the other way, and every later value of that row then
  follows that decision.  With ``masks`` the oracle takes those decisions and
  computes everything else itself; callers check first that the decisions
  they pass differ from the oracle's own only at such near-ties
  (``mask_disagreements``).
* AFDF: F[n, k] = exp(-2 pi i n k / N), F^{-1} its exact inverse conj(F)/N
  (Sec. 3); complex gradients follow the PyTorch convention
  grad = dL/dRe + i dL/dIm, i.e. g_x = g_y W^H.

Parity pins: see tests/test_oracle.py.  Every function here is pinned there
against something other than itself (a library DCT/FFT special case, closed
forms of the layer, a brute-force dense product, finite differences, and
torch autograd).
"""

from __future__ import annotations

import functools

import numpy as np

FLAG_PERM = 1
FLAG_RELU = 2
FLAG_COMPLEX = 4

_CHUNK = 512  # rows per dense product, only to bound memory


def _frozen(a: np.ndarray) -> np.ndarray:
    a.flags.writeable = False
    return a


@functools.lru_cache(maxsize=4)
def dct_matrix(N: int) -> np.ndarray:
    """Orthonormal DCT-II matrix C[n, k] (Sec. 4, definition of c_nk).

    c_nk = sqrt(2/N) * eps_k * cos(pi (2n+1) k / (2N)),  n, k in [0, N),
    eps_0 = 1/sqrt(2), eps_k = 1 otherwise.  Row vector x maps to x @ C.
    The integer argument (2n+1) k is kept reduced mod 4N (the cosine's
    period), so the angle is exact for wide rows, and the cosine is taken
    once for each of the 4N residues.  Row n + 1's arguments are row n's
    plus 2k.  (Cached: the result is read-only.)
    """
    k = np.arange(N, dtype=np.int64)
    eps = np.where(k == 0, 1.0 / np.sqrt(2.0), 1.0)
    cos_of_residue = np.cos(np.pi * np.arange(4 * N, dtype=np.float64) / (2.0 * N))
    C = np.empty((N, N))
    arg = k.copy()                       # (2n+1) k mod 4N for n = 0
    for n in range(N):
        C[n] = cos_of_residue[arg]
        arg += 2 * k                     # < 6N: one subtraction reduces it
        np.subtract(arg, 4 * N, out=arg, where=arg >= 4 * N)
    C *= np.sqrt(2.0 / N) * eps
    return _frozen(C)


@functools.lru_cache(maxsize=2)
def dft_matrix(N: int) -> np.ndarray:
    """Unnormalised DFT matrix F[n, k] = exp(-2 pi i n k / N) (Sec. 3, AFDF).

    The exponent is reduced mod N in integers before scaling so the angle is
    exact for large N.  (Cached: the result is read-only.)
    """
    n = np.arange(N, dtype=np.int64)[:, None]
    k = np.arange(N, dtype=np.int64)[None, :]
    return _frozen(np.exp(-2j * np.pi * ((n * k) % N).astype(np.float64) / N))


# Widths up to these use the dense matrices above; wider rows apply the same
# matrices through the library routines that tests/test_oracle.py equates
# with them (scipy's orthonormal DCT-II / DCT-III, numpy's FFT).  A real
# 16384^2 matrix takes 2.1 GB in float64; a complex one of that width would
# take 4.3 GB, so complex rows switch earlier.
DENSE_MAX_REAL = 16384
DENSE_MAX_COMPLEX = 8192


def dense_limit(complex_: bool) -> int:
    """Widest row the dense matrices serve (real or complex rows)."""
    return DENSE_MAX_COMPLEX if complex_ else DENSE_MAX_REAL


class _LibraryTransform:
    """The row-vector product h @ M for a DCT or DFT matrix M, evaluated by a
    library transform along the last axis.  Only __rmatmul__ is defined, so
    `h @ op` reads like the dense code it replaces."""

    __array_ufunc__ = None  # make numpy defer `ndarray @ op` to __rmatmul__

    def __init__(self, fn):
        self.fn = fn

    def __rmatmul__(self, h):
        return self.fn(np.asarray(h))


def _transforms(N: int, complex_: bool):
    """Return (T, Tinv, Tinv_H, T_H): the forward transform, its exact
    inverse, and the conjugate transposes the backward applies (row form).

    ACDC (Sec. 4): T = C, Tinv = C^T (C orthogonal), so Tinv_H = C, T_H = C^T.
    AFDF (Sec. 3): T = F, Tinv = conj(F) / N, so Tinv_H = F / N, T_H = conj(F).
    """
    if N <= dense_limit(complex_):
        if complex_:
            F = dft_matrix(N)
            T, Tinv = F, np.conj(F) / N
            return T, Tinv, np.conj(Tinv).T, np.conj(T).T
        # real: C^T is the exact inverse; views, no copies of a wide matrix
        C = dct_matrix(N)
        return C, C.T, C, C.T
    import scipy.fft
    if complex_:
        return (_LibraryTransform(lambda h: np.fft.fft(h, axis=-1)),
                _LibraryTransform(lambda h: np.fft.ifft(h, axis=-1)),
                _LibraryTransform(lambda h: np.fft.fft(h, axis=-1) / N),
                _LibraryTransform(lambda h: np.fft.ifft(h, axis=-1) * N))
    dct = _LibraryTransform(lambda h: scipy.fft.dct(h, type=2, norm="ortho", axis=-1))
    idct = _LibraryTransform(lambda h: scipy.fft.idct(h, type=2, norm="ortho", axis=-1))
    return dct, idct, dct, idct


def _check(x, A, D, perm, flags, B=None):
    x = np.asarray(x)
    A = np.asarray(A)
    D = np.asarray(D)
    if x.ndim != 2 or A.ndim != 2 or D.shape != A.shape or A.shape[1] != x.shape[1]:
        raise ValueError("shapes: x [B,N], A and D [K,N]")
    if B is not None and np.shape(B) != A.shape:
        raise ValueError("B must be [K,N]")
    if (flags & FLAG_COMPLEX) and (flags & FLAG_RELU):
        raise ValueError("ReLU is not defined for the complex variant")
    if flags & FLAG_PERM:
        perm = np.asarray(perm)
        if perm.shape != A.shape:
            raise ValueError("perm must be [K,N]")
        for k in range(perm.shape[0]):
            if not np.array_equal(np.sort(perm[k]), np.arange(A.shape[1])):
                raise ValueError(f"perm[{k}] is not a permutation")
    dt = np.complex128 if flags & FLAG_COMPLEX else np.float64
    Bd = np.zeros(A.shape, dt) if B is None else np.asarray(B).astype(dt)
    return x.astype(dt), A.astype(dt), D.astype(dt), perm, Bd


def _check_masks(masks, flags, K, shape):
    """ReLU decisions given as input: [K-1, B, N] bool (layer k's v_k > 0)."""
    if masks is None:
        return None
    if not flags & FLAG_RELU:
        raise ValueError("masks are ReLU decisions: they need FLAG_RELU")
    m = np.asarray(masks)
    if m.dtype != np.bool_ or m.shape != (K - 1,) + tuple(shape):
        raise ValueError("masks must be bool [K-1, B, N]")
    return m


def forward(x, A, D, perm=None, flags: int = 0, keep: bool = False, B=None, masks=None):
    """Cascade forward y = x prod_k [P_k] A_k T D_k T^{-1}  (eq. for AFDF_K in
    Sec. 3, made real in Sec. 4 as ACDC_K; permutations, ReLU and the D-domain
    biases as in Sec. 6.2).

    Per layer k (row vectors, Sec. 4 notation):
        u_k = z[:, perm[k]]          (if PERM)
        h1  = u_k * a_k              (x A)
        h2  = h1 @ T                 (x A C)
        h3  = h2 * d_k + b_k         (x A C D, plus the bias if B is given)
        v_k = h3 @ Tinv              (x A C D C^{-1})
        z   = max(v_k, 0)            (if RELU and k < K-1) else v_k

    With ``masks`` ([K-1, B, N] bool) the ReLU of layer k keeps v_k where
    masks[k] is true and zeroes it elsewhere, instead of deciding v_k > 0
    itself (the decisions of another evaluation; see the module docstring).

    Returns y, or (y, cache) with cache = dict(u=[...], h2=[...], v=[...]) of
    per-layer float64 arrays when ``keep`` is true.
    """
    x, A, D, perm, Bd = _check(x, A, D, perm, flags, B)
    K, N = A.shape
    masks = _check_masks(masks, flags, K, x.shape)
    T, Tinv, _, _ = _transforms(N, bool(flags & FLAG_COMPLEX))
    relu = bool(flags & FLAG_RELU)
    y = np.empty_like(x)
    cache = {"u": [np.empty_like(x) for _ in range(K)],
             "h2": [np.empty_like(x) for _ in range(K)],
             "v": [np.empty_like(x) for _ in range(K)]} if keep else None
    for r0 in range(0, x.shape[0], _CHUNK):
        z = x[r0:r0 + _CHUNK]
        for k in range(K):
            u = z[:, perm[k]] if flags & FLAG_PERM else z
            h1 = u * A[k]
            h2 = h1 @ T
            h3 = h2 * D[k] + Bd[k]
            v = h3 @ Tinv
            if relu and k < K - 1:
                z = np.maximum(v, 0.0) if masks is None else np.where(masks[k][r0:r0 + _CHUNK], v, 0.0)
            else:
                z = v
            if keep:
                cache["u"][k][r0:r0 + _CHUNK] = u
                cache["h2"][k][r0:r0 + _CHUNK] = h2
                cache["v"][k][r0:r0 + _CHUNK] = v
        y[r0:r0 + _CHUNK] = z
    return (y, cache) if keep else y


def backward(x, grad_y, A, D, perm=None, flags: int = 0, B=None, masks=None):
    """Analytic backward of the cascade (Sec. 4 derivative block, applied
    layer by layer in reverse; ReLU and permutation steps of Sec. 6.2).

    Real ACDC, per layer k from K-1 down to 0, with g = dL/dz_k:
        g    = g * (v_k > 0)                  (if RELU and k < K-1)
        gh3  = g @ C                          (dL/dh3 = C dL/dy in the paper's
                                               column form; row form g C)
        db_k = sum_rows gh3                   (the bias enters h3 additively)
        dd_k = sum_rows h2_k * gh3            (dL/dd = h2 . C dL/dy)
        gh1  = (gh3 * d_k) @ C^T              (C^{-1} d . C dL/dy)
        da_k = sum_rows u_k * gh1             (dL/da = x . C^{-1} d . C dL/dy)
        gu   = gh1 * a_k                      (dL/dx = a . C^{-1} d . C dL/dy)
        g[:, perm[k]] = gu                    (inverse of the gather)

    Complex AFDF (PyTorch convention g_x = g_y W^H):
        gh3 = g @ F / N, dd_k = sum conj(h2_k) gh3, gh1 = (gh3 conj(d_k)) @ conj(F),
        da_k = sum conj(u_k) gh1, gu = gh1 conj(a_k).

    With ``masks`` the ReLU decisions (v_k > 0 above) are taken from masks[k]
    instead, in the forward it recomputes and in the mask applied to g.

    Returns (grad_x [B,N], grad_A [K,N], grad_D [K,N]), and grad_B [K,N] as a
    fourth element when B is given; the parameter gradients are sums over the
    batch.  (B changes the stored h2 only through the forward values the
    backward recomputes: the ReLU masks of a biased cascade.)
    """
    x, A, D, perm, Bd = _check(x, A, D, perm, flags, B)
    masks = _check_masks(masks, flags, A.shape[0] if np.ndim(A) == 2 else 0, x.shape)
    cplx = bool(flags & FLAG_COMPLEX)
    gy = np.asarray(grad_y).astype(np.complex128 if cplx else np.float64)
    if gy.shape != x.shape:
        raise ValueError("grad_y must match x")
    K, N = A.shape
    # Backward transforms: row form of the transposed (conjugate-transposed
    # for AFDF) forward matrices: Tinv_H = C for ACDC, F / N for AFDF;
    # T_H = C^T for ACDC, conj(F) for AFDF.
    _, _, Tinv_H, T_H = _transforms(N, cplx)
    relu = bool(flags & FLAG_RELU)
    grad_x = np.empty_like(x)
    grad_A = np.zeros_like(A)
    grad_D = np.zeros_like(D)
    grad_B = np.zeros_like(D)
    for r0 in range(0, x.shape[0], _CHUNK):
        xs = x[r0:r0 + _CHUNK]
        ms = None if masks is None else masks[:, r0:r0 + _CHUNK]
        _, cache = forward(xs, A, D, perm, flags, keep=True, B=Bd, masks=ms)
        g = gy[r0:r0 + _CHUNK]
        for k in range(K - 1, -1, -1):
            if relu and k < K - 1:
                g = g * (cache["v"][k] > 0.0 if ms is None else ms[k])
            gh3 = g @ Tinv_H
            grad_B[k] += np.sum(gh3, axis=0)
            h2 = cache["h2"][k]
            grad_D[k] += np.sum((np.conj(h2) if cplx else h2) * gh3, axis=0)
            gh1 = (gh3 * (np.conj(D[k]) if cplx else D[k])) @ T_H
            u = cache["u"][k]
            grad_A[k] += np.sum((np.conj(u) if cplx else u) * gh1, axis=0)
            gu = gh1 * (np.conj(A[k]) if cplx else A[k])
            if flags & FLAG_PERM:
                g = np.empty_like(gu)
                g[:, perm[k]] = gu
            else:
                g = gu
        grad_x[r0:r0 + _CHUNK] = g
    if B is not None:
        return grad_x, grad_A, grad_D, grad_B
    return grad_x, grad_A, grad_D


def relu_decisions(cache, K: int) -> np.ndarray:
    """The oracle's own ReLU decisions v_k > 0, k < K-1, from a forward
    cache: [K-1, B, N] bool."""
    B, N = cache["v"][0].shape
    return np.array([cache["v"][k] > 0.0 for k in range(K - 1)], dtype=bool).reshape(K - 1, B, N)


def mask_disagreements(masks, cache, K: int, band: float) -> int:
    """Count the decisions in ``masks`` that differ from the oracle's own
    (forward cache computed with those masks) at a pre-ReLU value outside the
    near-tie band |v_k| < band * rms(v_k row).  Zero means every differing
    decision is one that rounding may legitimately take either way."""
    bad = 0
    for k in range(K - 1):
        v = cache["v"][k]
        rms = np.sqrt(np.mean(v * v, axis=1, keepdims=True))
        differ = np.asarray(masks[k]) != (v > 0.0)
        bad += int(np.count_nonzero(differ & (np.abs(v) >= band * rms)))
    return bad


def layer_matrix(a, d, complex_: bool = False) -> np.ndarray:
    """Dense matrix of one layer, A T D T^{-1} (Sec. 4 / Sec. 3); N small."""
    N = len(a)
    T, Tinv, _, _ = _transforms(N, complex_)
    dt = np.complex128 if complex_ else np.float64
    return np.diag(np.asarray(a, dt)) @ T @ np.diag(np.asarray(d, dt)) @ Tinv


def dense_operator(A, D, perm=None, flags: int = 0) -> np.ndarray:
    """Dense product W of a cascade without ReLU (eq. for AFDF_K, Sec. 3), so
    that y = x @ W.  Each gather u = z[:, p] is the permutation matrix with
    P[p[n], n] = 1.  Intended for N <= 64."""
    if flags & FLAG_RELU:
        raise ValueError("a cascade with ReLU is not a single matrix")
    A = np.asarray(A)
    K, N = A.shape
    cplx = bool(flags & FLAG_COMPLEX)
    W = np.eye(N, dtype=np.complex128 if cplx else np.float64)
    for k in range(K):
        if flags & FLAG_PERM:
            P = np.zeros((N, N))
            P[np.asarray(perm[k]), np.arange(N)] = 1.0
            W = W @ P
        W = W @ layer_matrix(A[k], D[k], cplx)
    return W


def flops_per_row_layer(N: int, complex_: bool = False) -> float:
    """Algorithmic flop count of one forward row-layer.

    ACDC: 4N + 5 N log2 N (Sec. 5, FFTW counting convention).
    AFDF: two complex N-point FFTs at 5 N log2 N each plus two complex
    diagonal products at 6N each.
    """
    lg = np.log2(N)
    if complex_:
        return 10.0 * N * lg + 12.0 * N
    return 4.0 * N + 5.0 * N * lg


def arithmetic_intensity(N: int) -> float:
    """Batched single-layer arithmetic intensity (4 + 5 log2 N) / 8 (Sec. 5)."""
    return (4.0 + 5.0 * np.log2(N)) / 8.0
