"""Seeded synthetic workloads for ACDC / AFDF cascades.

This module only draws random numbers: it holds none of the method's
arithmetic, so both the HIP path and the CPU oracle can take their inputs from
it without sharing any computation.

Recipe (numpy ``default_rng(seed)``; every draw in float64, then cast to
float32 / complex64 so that both sides see bit-identical inputs), in this
order: x, A, D, the permutations of layers 1..K-1 (``rng.permutation(N)``;
layer 0 keeps the identity, since the paper places permutations *between*
consecutive layers, Sec. 6.2), then the upstream gradient g_y.

* x ~ N(0, 1); for the ReLU cascades x = max(N(0,1), 0), standing in for the
  post-ReLU conv features that feed the cascade in Sec. 6.2.
* A, D ~ N(1, 0.1^2) i.i.d. (the initialisation Sec. 6.1 found to work for
  deep cascades).  For the complex variant the real parts follow N(1, 0.1^2)
  and the imaginary parts N(0, 0.1^2).
* g_y ~ N(0, 1) (real and imaginary parts independently for the complex
  variant).

The D-domain biases of the BIAS workloads (Sec. 6.2 adds them to the D
matrices and starts them at 0; a trained cascade holds small nonzero values)
come from a stream of their own, ``default_rng((seed, 8))``, so that the
draws above do not change: b ~ N(0, 0.1^2), float32, [K, N].
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

FLAG_PERM = 1
FLAG_RELU = 2
FLAG_COMPLEX = 4
FLAG_BIAS = 8
FLAG_ACCUMULATE = 16
FLAG_MULTIPASS = 32


@dataclass(frozen=True)
class Workload:
    name: str
    N: int
    K: int
    batch: int
    flags: int
    description: str

    @property
    def complex(self) -> bool:
        return bool(self.flags & FLAG_COMPLEX)


# The workloads: one single layer, a permuted cascade, the headline permuted
# ReLU cascade at N=4096, a non-power-of-two ReLU cascade at the width of a
# flattened 6x6x256 conv map, the complex AFDF cascade, a cascade wider than
# the fused kernels, and the headline cascade with D-domain biases.
WORKLOADS = {
    "acdc_n256_k1": Workload("acdc_n256_k1", 256, 1, 64, 0,
                             "single ACDC layer N=256, batch 64, fp32"),
    "acdc_n1024_k12_perm": Workload("acdc_n1024_k12_perm", 1024, 12, 4096, FLAG_PERM,
                                    "ACDC cascade N=1024 K=12 batch 4096, fp32, permutations"),
    "acdc_n4096_k12_perm_relu": Workload("acdc_n4096_k12_perm_relu", 4096, 12, 8192,
                                         FLAG_PERM | FLAG_RELU,
                                         "ACDC cascade N=4096 K=12 batch 8192, fp32, "
                                         "permutations + ReLU"),
    "acdc_n9216_k16_perm_relu": Workload("acdc_n9216_k16_perm_relu", 9216, 16, 1024,
                                         FLAG_PERM | FLAG_RELU,
                                         "ACDC cascade N=9216 K=16 batch 1024, fp32, "
                                         "permutations + ReLU"),
    "afdf_n4096_k8_perm": Workload("afdf_n4096_k8_perm", 4096, 8, 2048,
                                   FLAG_PERM | FLAG_COMPLEX,
                                   "complex AFDF cascade N=4096 K=8 batch 2048, complex64, "
                                   "permutations"),
    # past the fused kernels' width: the multi-pass path
    "acdc_n65536_k12_perm_relu": Workload("acdc_n65536_k12_perm_relu", 65536, 12, 512,
                                          FLAG_PERM | FLAG_RELU,
                                          "ACDC cascade N=65536 K=12 batch 512, fp32, permutations + ReLU "
                                          "(multi-pass)"),
    "afdf_n65536_k8_perm": Workload("afdf_n65536_k8_perm", 65536, 8, 256, FLAG_PERM | FLAG_COMPLEX,
                                    "complex AFDF cascade N=65536 K=8 batch 256, complex64, permutations "
                                    "(multi-pass)"),
    # the headline cascade with the D-domain biases of Sec. 6.2
    "acdc_n4096_k12_perm_relu_bias": Workload("acdc_n4096_k12_perm_relu_bias", 4096, 12, 8192,
                                              FLAG_PERM | FLAG_RELU | FLAG_BIAS,
                                              "ACDC cascade N=4096 K=12 batch 8192, fp32, "
                                              "permutations + ReLU + D-domain biases"),
}

HEADLINE = "acdc_n4096_k12_perm_relu"


def make_inputs(N: int, K: int, batch: int, flags: int, seed: int = 0,
                relu_input: bool | None = None):
    """Draw (x, A, D, perm, grad_y) following the recipe in the module doc.

    Returns numpy arrays: float32 (or complex64 when COMPLEX is set) for
    x, A, D, grad_y and int32 [K, N] for perm (identity rows when PERM is not
    set, so the array is always valid).
    """
    rng = np.random.default_rng(seed)
    cplx = bool(flags & FLAG_COMPLEX)
    if relu_input is None:
        relu_input = bool(flags & FLAG_RELU)
    if cplx:
        x = rng.standard_normal((batch, N)) + 1j * rng.standard_normal((batch, N))
        A = rng.normal(1.0, 0.1, (K, N)) + 1j * rng.normal(0.0, 0.1, (K, N))
        D = rng.normal(1.0, 0.1, (K, N)) + 1j * rng.normal(0.0, 0.1, (K, N))
    else:
        x = rng.standard_normal((batch, N))
        if relu_input:
            x = np.maximum(x, 0.0)
        A = rng.normal(1.0, 0.1, (K, N))
        D = rng.normal(1.0, 0.1, (K, N))
    perm = np.tile(np.arange(N, dtype=np.int32), (K, 1))
    if flags & FLAG_PERM:
        for k in range(1, K):
            perm[k] = rng.permutation(N).astype(np.int32)
    if cplx:
        gy = rng.standard_normal((batch, N)) + 1j * rng.standard_normal((batch, N))
    else:
        gy = rng.standard_normal((batch, N))
    dt = np.complex64 if cplx else np.float32
    return (x.astype(dt), A.astype(dt), D.astype(dt), perm, gy.astype(dt))


def make_bias(N: int, K: int, seed: int = 0) -> np.ndarray:
    """D-domain biases b ~ N(0, 0.1^2), float32 [K, N], from their own stream."""
    rng = np.random.default_rng((seed, 8))
    return rng.normal(0.0, 0.1, (K, N)).astype(np.float32)


def make_linreg(seed: int = 0, rows: int = 10000, N: int = 32):
    """Synthetic linear-regression data of Sec. 6.1: X [rows, N] and
    W_true [N, N] uniform on [0, 1), and the noise eps ~ N(0, 1e-4) (variance)
    of the targets Y = X W_true + eps, all float32.  Returns (X, W_true, eps);
    the caller forms Y."""
    rng = np.random.default_rng((seed, 61))
    X = rng.uniform(0.0, 1.0, (rows, N))
    W = rng.uniform(0.0, 1.0, (N, N))
    eps = rng.normal(0.0, 1e-2, (rows, N))
    return X.astype(np.float32), W.astype(np.float32), eps.astype(np.float32)


def make_workload(name: str, seed: int = 0, batch: int | None = None):
    """Inputs for one of the named workloads (optionally with another batch)."""
    w = WORKLOADS[name]
    return make_inputs(w.N, w.K, batch if batch is not None else w.batch, w.flags, seed)
