"""Benchmark: ACDC cascade forward + backward on one MI355X.

A step is one training pass of the whole cascade over one batch: the forward
kernel (which also stores what the backward needs) followed by the backward kernel and
the fixed-order reduction of dL/da, dL/dd.  Inputs are synthetic and seeded
(paper_1511_05946_amd.workloads) and already resident in HBM when timing
starts.

Prints ONE JSON line (plus diagnostics on stderr):
  value      rows*layers/s = batch*K / (seconds per step)
  roofline   the dominant kernel (backward cascade) against the fp32 vector
             peak: algorithmic flops per launch / measured launch time
  cpu_baseline  the fp64 oracle on a bounded sample of the same workload
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "ACDC rows·layers/sec (fwd+bwd) at N=4096,K=12; % of HBM/fp32 roofline"
UNIT = "rows·layers/s"
PEAK_FP32_TFLOPS = 157.3     # MI355X fp32 vector peak (256 CU x 2.4 GHz x 256 flop/clk)
PEAK_HBM_GBPS = 8000.0


def flops_row_layer(N: int, complex_: bool) -> float:
    # Sec. 5 count: 4N + 5N log2 N per row-layer (FFTW convention); AFDF: two
    # complex N-point FFTs and two complex diagonals.
    lg = math.log2(N)
    return (10 * N * lg + 12 * N) if complex_ else (4 * N + 5 * N * lg)


def recorded_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the rocprofv3 FETCH_SIZE /
    WRITE_SIZE record in profiles/, scaled by the copy calibration stored with
    it; None when there is no record or the kernel sources changed since the
    counters were taken."""
    from paper_1511_05946_amd.build import source_digest
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_digest") != source_digest() or kernel not in rec.get("kernels", {}):
        return None
    k = rec["kernels"][kernel]
    return (k["fetch_kib"] * rec["fetch_scale"] + k["write_kib"] * rec["write_scale"]) * 1024.0


def cpu_baseline(w, seed: int, budget_s: float = 20.0, max_rows: int = 2048):
    """Time the oracle (forward + analytic backward, fp64, as it stands) on the
    first rows of the workload.  The sample grows from 8 rows until one call
    fills half of budget_s (so the reported call takes about 10-20 s), up to
    max_rows rows or the whole batch; at the widths up to 9216 that is at
    least the first 512 rows.  The last call is the one reported.  The dense
    matrix is built before timing starts."""
    import numpy as np  # noqa: F401
    from threadpoolctl import threadpool_info

    from oracle import acdc_oracle as O
    from paper_1511_05946_amd.workloads import FLAG_BIAS, make_bias, make_inputs

    x, A, D, perm, gy = make_inputs(w.N, w.K, min(w.batch, max_rows), w.flags, seed)
    bias = make_bias(w.N, w.K, seed) if w.flags & FLAG_BIAS else None
    dense = w.N <= O.dense_limit(w.complex)
    if dense:
        (O.dft_matrix if w.complex else O.dct_matrix)(w.N)

    def run(rows):
        t0 = time.perf_counter()
        O.forward(x[:rows], A, D, perm, w.flags & 7, B=bias)
        O.backward(x[:rows], gy[:rows], A, D, perm, w.flags & 7, B=bias)
        return time.perf_counter() - t0

    rows = min(8, x.shape[0])
    t_total = run(rows)
    # small samples run below the oracle's rate (each product re-reads the
    # whole matrix), so grow the sample until it fills half the budget
    while rows < x.shape[0] and t_total < 0.5 * budget_s:
        rows = int(min(x.shape[0], max(2 * rows, rows * budget_s / max(t_total, 1e-9))))
        t_total = run(rows)
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {"value": rows * w.K / t_total, "unit": UNIT, "cores": int(threads), "kind": "oracle",
            "blas_threads": int(threads), "affinity_cores": len(os.sched_getaffinity(0)),
            "sample": f"first {rows} of {w.batch} rows, full N={w.N}, K={w.K}, fwd + bwd, fp64 oracle "
                      + ("(O(N^2) dense matrices, built before timing)" if dense
                         else "(library DCT/FFT past the dense limit)")
                      + f", {t_total:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--recompute", action="store_true",
                    help="backward recomputes the layer inputs instead of using the forward's")
    ap.add_argument("--multipass", action="store_true",
                    help="run the layers through the multi-pass (HBM) path instead of the fused kernels")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--flush-mb", type=int, default=0,
                    help="write this many MB between steps (evicts the 256 MB Infinity Cache); value and "
                         "ms_per_step then come from per-step HIP events, without the flush")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 256 MiB device copy (known bytes) so that profiler "
                         "byte counters can be scaled against it")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU only (asked for --gpus {args.gpus}); "
              "the cascade shards over rows with one all-reduce of dL/da, dL/dd, "
              "which is not built here.", file=sys.stderr)
        sys.exit(2)

    import ctypes

    import torch

    import paper_1511_05946_amd.acdc as acdc
    from paper_1511_05946_amd._lib import lib
    from paper_1511_05946_amd.workloads import FLAG_BIAS, HEADLINE, WORKLOADS, make_bias, make_inputs

    w = WORKLOADS[args.workload or HEADLINE]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copy calibration: 3 copies of {src.numel() * 4} bytes read + written",
              file=sys.stderr)
        del src, dst
    x, A, D, perm, gy = make_inputs(w.N, w.K, w.batch, w.flags, args.seed)
    t = lambda a: torch.from_numpy(a).to(dev)
    xt, At, Dt, pt, gyt = t(x), t(A), t(D), t(perm), t(gy)
    bt = t(make_bias(w.N, w.K, args.seed)) if w.flags & FLAG_BIAS else None
    fl = w.flags & ~acdc.FLAG_COMPLEX
    if args.multipass:
        fl |= acdc.FLAG_MULTIPASS
    # the fused kernels cover ACDC widths up to 32768 and AFDF up to 16384;
    # wider rows run multi-pass
    multipass = args.multipass or w.N > (16384 if w.complex else 32768)
    acdc.prepare(w.N, fl | (acdc.FLAG_COMPLEX if w.complex else 0))
    y = torch.empty_like(xt)
    saved = acdc.alloc_saved(xt, w.K, fl)

    def step():
        if args.recompute:
            acdc.forward(xt, At, Dt, pt, fl, out=y, bias=bt)
            return acdc.backward(xt, gyt, At, Dt, pt, fl, saved=None, bias=bt)
        acdc.forward(xt, At, Dt, pt, fl, out=y, saved=saved, bias=bt)
        return acdc.backward(xt, gyt, At, Dt, pt, fl, saved=saved, bias=bt)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    flush = torch.empty((args.flush_mb << 20) // 4, dtype=torch.float32, device=dev) if args.flush_mb > 0 else None
    L = lib()
    L.acdc_profile_enable(1)
    ms = (ctypes.c_double * 3)()
    cnt = (ctypes.c_int64 * 3)()
    L.acdc_profile_read(ms, cnt)  # clear
    # per-step HIP events on the stream the library launches on (torch's current one)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        if flush is not None:
            flush.fill_(float(i))
        ev[i][0].record()
        step()
        ev[i][1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    rc = L.acdc_profile_read(ms, cnt)
    L.acdc_profile_enable(0)
    if rc != 0:
        raise RuntimeError(f"acdc_profile_read failed: {rc}")
    step_ms = sorted(a.elapsed_time(b) for a, b in ev)

    ms_step = sum(step_ms) / args.steps if flush is not None else (t1 - t0) * 1e3 / args.steps
    value = w.batch * w.K / (ms_step * 1e-3)
    kern = {name: {"avg_ms": ms[i] / max(cnt[i], 1), "launches": int(cnt[i])}
            for i, name in enumerate(("forward", "backward", "reduce"))}
    fwd_launches_per_step = cnt[0] / args.steps
    f_rl = flops_row_layer(w.N, w.complex)
    # dominant kernel: the backward cascade; its algorithmic work is one pass
    # of the layer transform per row-layer, like the forward (Sec. 5).
    bwd_ms = kern["backward"]["avg_ms"]
    bwd_flops = w.batch * w.K * f_rl
    achieved = bwd_flops / (bwd_ms * 1e-3) / 1e12
    fwd_ms = kern["forward"]["avg_ms"]
    fwd_achieved = w.batch * w.K * f_rl / (fwd_ms * 1e-3) / 1e12
    roof = {"bound": "alu", "achieved": round(achieved, 3), "peak": PEAK_FP32_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_TFLOPS, 4),
            "traffic": None if multipass else recorded_traffic(w.name, "k_real_bwd" if not w.complex else "k_cplx_bwd"),
            "kernel": ("multi-pass backward (whole launch sequence)" if multipass
                       else "k_real_bwd" if not w.complex else "k_cplx_bwd"),
            "kernel_avg_ms": round(bwd_ms, 4),
            "algorithmic_flops_per_launch": bwd_flops}
    # fraction of the whole-step roofline (fwd+bwd algorithmic flops at peak)
    step_flops = 2 * w.batch * w.K * f_rl
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": UNIT, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "c64" if w.complex else "f32",
        "data": "synthetic (seeded; x ~ relu(N(0,1)), A,D ~ N(1,0.1^2), random permutations"
                + (", D-domain biases ~ N(0,0.1^2))" if bt is not None else ")"),
        "config": {"workload": w.name, "N": w.N, "K": w.K, "batch": w.batch,
                   "flags": w.flags, "parallelism": "single GPU",
                   "backward": "recompute" if args.recompute else "saved layer inputs",
                   "path": "multi-pass" if multipass else "fused"},
        "roofline": roof,
        "step_roofline_frac": round(step_flops / (ms_step * 1e-3) / 1e12 / PEAK_FP32_TFLOPS, 4),
        "kernels": {k: {"avg_ms": round(v["avg_ms"], 4), "launches": v["launches"]} for k, v in kern.items()},
        "forward_tflops": round(fwd_achieved, 3),
        "step_ms_median": round(step_ms[len(step_ms) // 2], 4),
        "step_ms_min": round(step_ms[0], 4),
        "flush_mb_between_steps": args.flush_mb,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.seed)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    print(f"[bench] fwd kernel {fwd_ms:.3f} ms ({fwd_launches_per_step:.0f}/step), bwd kernel {bwd_ms:.3f} ms, "
          f"reduce {kern['reduce']['avg_ms']:.3f} ms, step {ms_step:.3f} ms", file=sys.stderr)


if __name__ == "__main__":
    main()
