"""Single ACDC layer against a dense linear layer, forward and backward, at
batch 128 over N = 128 ... 16384 (the comparison of Sec. 5, Fig. 2).

    python -m paper_1511_05946_amd.sweep [--batch 128] [--reps 50] [--sizes 128,256,...]

ACDC: one layer y = x A C D C^{-1} through the library (forward: acdc_forward;
backward: acdc_backward, which recomputes the layer's D input from x as the
paper's backward does).  Dense: y = x W with torch.mm on the same device
(rocBLAS / hipBLASLt fp32 GEMM), backward dX = dY W^T and dW = X^T dY.  Both
sides run in fp32.  Each call is timed twice, with HIP events around `reps`
back-to-back calls (median of 5 groups):

* eager: the calls as a Python caller makes them (host launch overhead
  included; at batch 128 it dominates both sides below N = 4096);
* graph: the same calls captured once into a HIP graph and replayed, which
  leaves the device time.  Every replay's outputs are checked bitwise
  against the eager outputs.

Prints one JSON line per width, then a markdown table.

Algorithmic flops per row: ACDC 4N + 5N log2 N per pass (Sec. 5); dense 2N^2
forward and 4N^2 backward.
"""

from __future__ import annotations

import argparse
import json
import math
import statistics

import torch

from . import acdc
from .workloads import make_inputs


def _time(fn, reps: int) -> float:
    """Median over 5 groups of the mean per-call time (ms) of `reps` calls."""
    fn()
    torch.cuda.synchronize()
    groups = []
    for _ in range(5):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        b.synchronize()
        groups.append(a.elapsed_time(b) / reps)
    return statistics.median(groups)


def _time_graph(fn, reps: int, outputs) -> float:
    """The same as _time on a HIP graph of `reps` calls; after every replay
    the outputs must equal the eager result bit for bit."""
    fn()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outputs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    groups = []
    for _ in range(5):
        for o in outputs:
            o.zero_()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        g.replay()
        b.record()
        b.synchronize()
        groups.append(a.elapsed_time(b) / reps)
        for o, r in zip(outputs, ref):
            if not torch.equal(o, r):
                raise RuntimeError("graph replay differs from the eager result")
    return statistics.median(groups)


def run(batch: int, sizes, reps: int):
    dev = torch.device("cuda:0")
    rows = []
    for N in sizes:
        x, A, D, _, gy = make_inputs(N, 1, batch, 0, seed=N)
        t = lambda a: torch.from_numpy(a).to(dev)
        xt, At, Dt, gyt = t(x), t(A), t(D), t(gy)
        acdc.prepare(N, 0)
        y = torch.empty_like(xt)
        gxa = torch.empty_like(xt)
        grads = (torch.empty_like(At), torch.empty_like(Dt))
        f_acdc = lambda: acdc.forward(xt, At, Dt, None, 0, out=y)
        b_acdc = lambda: acdc.backward(xt, gyt, At, Dt, None, 0, grads=grads, out=gxa)
        W = torch.randn(N, N, device=dev, generator=torch.Generator(dev).manual_seed(N)) / math.sqrt(N)
        yd = torch.empty(batch, N, device=dev)
        gx = torch.empty(batch, N, device=dev)
        gW = torch.empty(N, N, device=dev)
        f_dense = lambda: torch.mm(xt, W, out=yd)

        def b_dense():
            torch.mm(gyt, W.t(), out=gx)
            torch.mm(xt.t(), gyt, out=gW)

        r = {"N": N, "batch": batch,
             "acdc_fwd_ms": _time(f_acdc, reps), "acdc_bwd_ms": _time(b_acdc, reps),
             "dense_fwd_ms": _time(f_dense, reps), "dense_bwd_ms": _time(b_dense, reps),
             "acdc_fwd_graph_ms": _time_graph(f_acdc, reps, [y]),
             "acdc_bwd_graph_ms": _time_graph(b_acdc, reps, [gxa, *grads]),
             "dense_fwd_graph_ms": _time_graph(f_dense, reps, [yd]),
             "dense_bwd_graph_ms": _time_graph(b_dense, reps, [gx, gW])}
        f_layer = batch * (4 * N + 5 * N * math.log2(N))
        r["acdc_fwd_gflops"] = f_layer / (r["acdc_fwd_ms"] * 1e-3) / 1e9
        r["dense_fwd_gflops"] = 2.0 * batch * N * N / (r["dense_fwd_ms"] * 1e-3) / 1e9
        r["acdc_fwd_graph_gflops"] = f_layer / (r["acdc_fwd_graph_ms"] * 1e-3) / 1e9
        r["dense_fwd_graph_gflops"] = 2.0 * batch * N * N / (r["dense_fwd_graph_ms"] * 1e-3) / 1e9
        r["speedup_fwd"] = r["dense_fwd_ms"] / r["acdc_fwd_ms"]
        r["speedup_bwd"] = r["dense_bwd_ms"] / r["acdc_bwd_ms"]
        r["speedup_fwd_graph"] = r["dense_fwd_graph_ms"] / r["acdc_fwd_graph_ms"]
        r["speedup_bwd_graph"] = r["dense_bwd_graph_ms"] / r["acdc_bwd_graph_ms"]
        rows.append(r)
        print(json.dumps({k: (round(v, 5) if isinstance(v, float) else v) for k, v in r.items()}), flush=True)
        del W, gW
        torch.cuda.empty_cache()
    print()
    print("| N | ACDC fwd | ACDC bwd | dense fwd | dense bwd | dense/ACDC fwd | dense/ACDC bwd | "
          "graph: ACDC fwd | ACDC bwd | dense fwd | dense bwd | dense/ACDC fwd | dense/ACDC bwd |")
    print("|---" * 13 + "|")
    us = lambda ms: f"{ms * 1e3:.1f} µs"
    for r in rows:
        print(f"| {r['N']} | {us(r['acdc_fwd_ms'])} | {us(r['acdc_bwd_ms'])} | {us(r['dense_fwd_ms'])} | "
              f"{us(r['dense_bwd_ms'])} | {r['speedup_fwd']:.1f}x | {r['speedup_bwd']:.1f}x | "
              f"{us(r['acdc_fwd_graph_ms'])} | {us(r['acdc_bwd_graph_ms'])} | {us(r['dense_fwd_graph_ms'])} | "
              f"{us(r['dense_bwd_graph_ms'])} | {r['speedup_fwd_graph']:.1f}x | {r['speedup_bwd_graph']:.1f}x |")
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--batch", type=int, default=128)
    ap.add_argument("--reps", type=int, default=50)
    ap.add_argument("--sizes", default=",".join(str(1 << p) for p in range(7, 15)))
    a = ap.parse_args()
    torch.backends.cuda.matmul.allow_tf32 = False
    run(a.batch, [int(s) for s in a.sizes.split(",")], a.reps)


if __name__ == "__main__":
    main()
