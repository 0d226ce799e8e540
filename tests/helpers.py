"""Shared test helpers: the parity metric and the ReLU-margin row filter."""

from __future__ import annotations

import numpy as np

# Max relative error per output (fp32, K <= 16) and for the complex variant.
TOL_REAL = 1e-4
TOL_COMPLEX = 2e-4
# ReLU decisions closer than DELTA * rms(row) to zero may legitimately differ
# between fp32 and fp64, and one flipped mask bit changes that row's gradient.
RELU_DELTA = 1e-5


def rel_err(got, ref) -> float:
    """max_i |got_i - ref_i| / max(|ref_i|, rms(ref over the group)), groups =
    rows (last axis).  Handles complex arrays through their modulus."""
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    ref2 = ref.reshape(-1, ref.shape[-1]) if ref.ndim > 1 else ref.reshape(1, -1)
    got2 = got.reshape(ref2.shape)
    rms = np.sqrt(np.mean(np.abs(ref2) ** 2, axis=1, keepdims=True))
    den = np.maximum(np.abs(ref2), rms)
    den = np.where(den == 0, 1.0, den)
    err = np.abs(got2.astype(np.complex128 if np.iscomplexobj(ref2) else np.float64) - ref2) / den
    if not np.all(np.isfinite(err)):
        return float("inf")
    return float(err.max())


def relu_safe_rows(cache_v, K: int, delta: float = RELU_DELTA) -> np.ndarray:
    """Rows whose pre-ReLU values |v_k| stay above delta * rms(v_k row) for
    every layer k < K-1 (oracle forward cache)."""
    ok = None
    for k in range(K - 1):
        v = cache_v[k]
        rms = np.sqrt(np.mean(v * v, axis=1, keepdims=True))
        row_ok = np.all(np.abs(v) >= delta * rms, axis=1)
        ok = row_ok if ok is None else ok & row_ok
    if ok is None:
        ok = np.ones(cache_v[0].shape[0], dtype=bool)
    return ok
