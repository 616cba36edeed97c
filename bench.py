#!/usr/bin/env python3
"""Training-throughput benchmark of the Polyglot window-LM SGD step on one MI355X.

One "step" is the whole hot path over one batch: gather, tanh hidden layer
and scores for the true and the corrupted windows, hinge loss, backward, the
sorted-segment embedding scatter-add and the dense SGD update.  Inputs are
seeded synthetic Zipf word windows, staged in device memory before timing.

Prints ONE JSON line (rank 0) with windows/s, the roofline of the dominant
kernel (per-kernel HIP events on the library's stream) and the CPU oracle
timed on the host as a baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, published
MFMA_F32_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix, published


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="sweep_1024")
    ap.add_argument("--mode", choices=("sorted", "atomic"), default="sorted")
    ap.add_argument("--graph", action="store_true",
                    help="replay the timed steps as one captured HIP graph")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    return ap.parse_args()


def kernel_model(w, B, U, n_parts):
    """Algorithmic bytes and flops of one launch of each kernel of a step."""
    d, win, H, K = w.d, w.win, w.H, w.K
    N = B * (win + 1)
    fwd_bytes = B * ((win + 1) * 4 + (win + 1) * d * 4 + 3 * H * 4) + H * K * 4
    fwd_flops = B * 4 * H * (K + d)
    upd_bytes = N * (8 + 4 * H) + U * 2 * d * 4 + 2 * H * K * 4
    upd_flops = 0
    sort_bytes = N * 16
    return {
        "fwdbwd": (fwd_bytes, fwd_flops),
        "update": (upd_bytes, upd_flops),
        "sort": (sort_bytes, 0),
    }


def cpu_baseline(w, seconds):
    import numpy as np
    import oracle
    import workloads
    p = workloads.init_params(w)
    steps = 0
    t0 = time.perf_counter()
    busy = 0.0
    while busy < seconds:
        win, cor = workloads.batch(w, steps, w.B)
        a = time.perf_counter()
        oracle.train_step(p, win, cor, w.lr)
        busy += time.perf_counter() - a
        steps += 1
    del t0
    return {
        "value": round(w.B * steps / busy, 1),
        "unit": "windows/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"first {steps} steps of {w.name} (B={w.B}), float32-storage float64-arithmetic "
                  f"C++ oracle, single thread, {busy:.1f} s of step time",
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); this build has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_1404_1521_amd as pg
    import workloads

    w = workloads.PRESETS[args.workload]
    B, K, Wm = w.B, args.steps, args.warmup
    mode = pg.SCATTER_SORTED if args.mode == "sorted" else pg.SCATTER_ATOMIC
    torch.cuda.set_device(0)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        p = workloads.init_params(w)
        pd = {k: torch.from_numpy(v).cuda() for k, v in p.items()}
        nb = Wm + 2 * K
        wins = np.empty((nb, B, w.win), np.int32)
        cors = np.empty((nb, B), np.int32)
        for s in range(nb):
            wins[s], cors[s] = workloads.batch(w, s, B)
        U = int(np.mean([np.unique(np.concatenate([wins[s].ravel(), cors[s]])).size
                         for s in range(min(nb, 8))]))
        dwin = torch.from_numpy(wins).cuda()
        dcor = torch.from_numpy(cors).cuda()
        losses = torch.zeros(nb, device="cuda")
        ctx = pg.Context(w.V, w.d, w.win, w.H, max_batch=B, scatter_mode=mode, stream=stream)

        def run(lo, hi):
            if args.graph:
                ctx.train_steps(pd, dwin[lo:hi], dcor[lo:hi], w.lr, losses[lo:hi])
            else:
                for s in range(lo, hi):
                    ctx.train_step(pd, dwin[s], dcor[s], w.lr, losses[s:s + 1])

        # warmup (with --graph this also captures the graph of the timed steps)
        for s in range(Wm):
            ctx.train_step(pd, dwin[s], dcor[s], w.lr, losses[s:s + 1])
        if args.graph:
            run(Wm, Wm + K)
        stream.synchronize()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        run(Wm, Wm + K)
        e1.record(stream)
        stream.synchronize()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = e0.elapsed_time(e1)
        if ctx.status() != pg.OK:
            raise RuntimeError("device error flag raised during the benchmark")

        # per-kernel durations: the next K steps with event brackets on the library stream
        ctx.set_timing(True)
        for s in range(Wm + K, Wm + 2 * K):
            ctx.train_step(pd, dwin[s], dcor[s], w.lr, losses[s:s + 1])
        kt = ctx.kernel_times()
        ctx.set_timing(False)
        lh = losses.cpu().numpy()
        if not np.all(np.isfinite(lh)):
            raise RuntimeError("non-finite loss")

    n_parts = min(-(-B // 16), 512)
    model = kernel_model(w, B, U, n_parts)
    per = {k: (v[0] / v[1] if v[1] else 0.0, v[1]) for k, v in kt.items() if v[1]}
    dom = max(per, key=lambda k: per[k][0] * per[k][1])
    dms, dlaunch = per[dom]
    nbytes, nflops = model.get(dom, (0, 0))
    intensity = nflops / nbytes if nbytes else 0.0
    if nflops and intensity > MFMA_F32_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        ach = nflops / (dms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 3), "peak": MFMA_F32_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / MFMA_F32_PEAK_TFLOPS, 5), "traffic": None}
    else:
        ach = nbytes / (dms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 5), "traffic": None}
    roof["kernel"] = dom
    roof["avg_launch_us"] = round(dms * 1e3, 3)
    roof["kernels_us"] = {k: round(v[0] * 1e3, 3) for k, v in per.items()}

    value = B * K / (ms * 1e-3)
    out = {
        "metric": "training windows/sec (fwd+bwd+update) at V=100k,d=64,win=5,B=1024; HBM GB/s",
        "value": round(value, 1),
        "unit": "windows/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": round(ms / K, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: V={w.V} d={w.d} win={w.win} H={w.H} B={B} "
                               f"ids Zipf({w.zipf_s}) corrupt uniform lr={w.lr} "
                               f"scatter={args.mode}{' graph' if args.graph else ''}",
                   "global_batch": B, "parallelism": "single-gpu"},
        "roofline": roof,
        "wall_s": round(wall, 4),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
