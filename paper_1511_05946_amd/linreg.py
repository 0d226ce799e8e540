"""Recovering a dense linear operator with ACDC_K by stochastic gradient
descent: the synthetic linear-regression experiment of Sec. 6.1.

    python -m paper_1511_05946_amd.linreg [--K 1,2,4,8,16,32] [--steps 3000]

Problem (Sec. 6.1): Y = X W_true + eps with X [10000, 32] and W_true [32, 32]
uniform on [0, 1) and eps ~ N(0, 1e-4).  The model is an ACDC cascade of K
layers (no permutations, no ReLU), y = x prod_k A_k C D_k C^{-1}, trained on
the mean squared error over minibatches of 100 rows, forward and backward
through the library (acdc_cascade).  Two initialisations of the diagonals
(Sec. 6.1, Fig. 3):

* identity: A, D = 1 + N(0, 0.1^2) -- the paper's recommendation for deep
  cascades (identity plus a small perturbation that breaks symmetries);
* small: A, D ~ N(0, (1e-3)^2) -- a standard small-weight initialisation.

The optimiser is Adam (learning rate 1e-2): Sec. 6.1 names SGD without its
settings, and plain momentum SGD at a rate that makes progress at K = 1
diverges at K >= 16 here.  The dense reference is the least-squares
operator (the noise floor, 1e-4).  Prints one JSON line per (init, K), then
a markdown table of the final losses on all rows.
"""

from __future__ import annotations

import argparse
import json

import torch

from . import acdc
from .workloads import make_linreg


def init_params(K: int, N: int, init: str, seed: int, device):
    g = torch.Generator(device="cpu").manual_seed(seed)
    mean, std = (1.0, 0.1) if init == "identity" else (0.0, 1e-3)
    A = (mean + std * torch.randn(K, N, generator=g)).to(device)
    D = (mean + std * torch.randn(K, N, generator=g)).to(device)
    return A.requires_grad_(True), D.requires_grad_(True)


def full_loss(X, Y, A, D) -> float:
    with torch.no_grad():
        y, _ = acdc.forward(X, A.detach().contiguous(), D.detach().contiguous(), None, 0)
        return float(((y - Y) ** 2).mean())


def train(X, Y, K: int, init: str, steps: int = 3000, lr: float = 1e-2, batch: int = 100, seed: int = 0,
          log_every: int = 0):
    """Train ACDC_K on (X, Y); returns (A, D, [(step, full-data loss), ...])."""
    N = X.shape[1]
    A, D = init_params(K, N, init, seed + K, X.device)
    opt = torch.optim.Adam([A, D], lr=lr)
    g = torch.Generator(device="cpu").manual_seed(seed)
    hist = [(0, full_loss(X, Y, A, D))]
    for step in range(1, steps + 1):
        idx = torch.randint(0, X.shape[0], (batch,), generator=g).to(X.device)
        pred = acdc.acdc_cascade(X[idx].contiguous(), A, D, None, 0)
        loss = ((pred - Y[idx]) ** 2).mean()
        opt.zero_grad(set_to_none=True)
        loss.backward()
        opt.step()
        if log_every and step % log_every == 0:
            hist.append((step, full_loss(X, Y, A, D)))
    if not log_every or hist[-1][0] != steps:
        hist.append((steps, full_loss(X, Y, A, D)))
    return A, D, hist


def problem(seed: int, device):
    X, W, eps = make_linreg(seed)
    Xt = torch.from_numpy(X).to(device)
    Yt = Xt @ torch.from_numpy(W).to(device) + torch.from_numpy(eps).to(device)
    return Xt, Yt


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--K", default="1,2,4,8,16,32")
    ap.add_argument("--steps", type=int, default=3000)
    ap.add_argument("--lr", type=float, default=1e-2)
    ap.add_argument("--seed", type=int, default=0)
    a = ap.parse_args()
    dev = torch.device("cuda:0")
    X, Y = problem(a.seed, dev)
    sol = torch.linalg.lstsq(X.double().cpu(), Y.double().cpu()).solution
    dense = float(((X.double().cpu() @ sol - Y.double().cpu()) ** 2).mean())
    print(json.dumps({"model": "dense least squares", "loss": dense}), flush=True)
    rows = []
    for init in ("identity", "small"):
        for K in [int(k) for k in a.K.split(",")]:
            _, _, hist = train(X, Y, K, init, a.steps, a.lr, seed=a.seed, log_every=max(a.steps // 10, 1))
            rows.append((init, K, hist[0][1], hist[-1][1]))
            print(json.dumps({"init": init, "K": K, "loss_start": hist[0][1], "loss_end": hist[-1][1],
                              "history": hist}), flush=True)
    print()
    print(f"| init | K | loss at start | loss after {a.steps} steps |")
    print("|---|---|---|---|")
    for init, K, l0, l1 in rows:
        print(f"| {init} | {K} | {l0:.4g} | {l1:.4g} |")
    print(f"| dense least squares | — | — | {dense:.3g} |")


if __name__ == "__main__":
    main()
