#!/usr/bin/env python3
"""Training-throughput benchmark of the Polyglot window-LM SGD step on one MI355X.

One "step" is the whole hot path over one batch: gather, tanh hidden layer
and scores for the true and the corrupted windows, hinge loss, backward, the
sorted-segment embedding scatter-add and the dense SGD update.  Inputs are
seeded synthetic Zipf word windows, staged in device memory before timing.

Prints ONE JSON line with windows/s, the roofline of the dominant kernel of
the step (per-kernel HIP events on the library's stream), the standalone
gather and scatter-add kernels at their full sizes against the HBM roofline,
and the CPU oracle timed on the host as a baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

COUNTERS = os.path.join(ROOT, "profiles", "hbm_counters_{}.md")
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
F32_MATRIX_PEAK_TFLOPS = 157.3  # MI355X dense fp32 MFMA, published
F32_VECTOR_PEAK_TFLOPS = 157.3  # 256 CU x 4 SIMD x 64 lanes x 2 flop (FMA) x 2.4 GHz


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="sweep_1024")
    ap.add_argument("--batch", type=int, default=0,
                    help="windows per step instead of the workload's own (same model and inputs)")
    ap.add_argument("--mode", choices=("sorted", "atomic"), default="sorted")
    ap.add_argument("--eager", action="store_true",
                    help="one library call per step instead of one captured graph of all steps")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernels", action="store_true",
                    help="skip the standalone gather / scatter-add measurements")
    ap.add_argument("--only-kernels", action="store_true",
                    help="run only the standalone gather / scatter-add measurements (no step, "
                         "no JSON line): isolates their dispatches under a counter profiler")
    ap.add_argument("--convergence", action="store_true",
                    help="batch size vs convergence on the planted synthetic task (one JSON line)")
    ap.add_argument("--conv-budget", type=int, default=8_000_000,
                    help="training windows per run of the convergence study")
    ap.add_argument("--conv-target", type=float, default=0.05,
                    help="held-out ranking error that ends a run of the convergence study")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 5 plain device copies of MIB MiB (calibrates the HBM byte "
                         "counters: each copy reads and writes exactly MIB MiB) and exit")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# Algorithmic bytes and flops of each kernel, from the batch itself.

def _hp(H):
    return -(-H // 16) * 16


def seg_chunk(N):
    """Sorted entries per wave in the segmented update (mirrors the library's choice)."""
    return 16 if N <= 131072 else 64


def batch_structure(wins, cors, ch):
    """Distinct rows U, rows whose sorted entries span several chunks, and the
    chunk partials those rows leave (entry order = window-major, corrupt last)."""
    import numpy as np
    B, win = wins.shape
    keys = np.concatenate([wins, cors[:, None]], axis=1).ravel()
    order = np.argsort(keys, kind="stable")
    sk = keys[order]
    heads = np.flatnonzero(np.r_[True, sk[1:] != sk[:-1]])
    ends = np.r_[heads[1:], sk.size]
    cs, ce = heads // ch, (ends - 1) // ch
    long_rows = cs != ce
    return {"U": int(heads.size), "long_rows": int(long_rows.sum()),
            "partials": int((ce - cs + 1)[long_rows].sum())}


def step_model(w, B, st, passes, n_parts):
    """({kernel: (bytes, flops, engine)}, {kernel: overhead bytes}) of one step.

    The first map holds the method's own bytes and flops per step: what the
    operation must read, write and compute whatever the implementation.  The
    second holds the traffic this implementation adds on top (the dense
    gradient partials that one kernel writes and the next reads back), which
    is reported beside the roofline, never inside it.

    Hidden layers of at most 64 units (one fused kernel):
    fwdbwd: ids + every window row and corrupt row read once (the gather),
      the per-entry gradient rows G written ((win+1) rows of d floats per
      window), W1 read once: (win+1)(4 + 8d) B per window, 3,096 B at d 64,
      window 5; flops = forward 2HK + 2Hd (corrupted centre block), dW1
      2HK + 2Hd, G (win+1) 2Hd per window: 73,728 at H 32 (plus O(H)
      elementwise work, not counted).  Overhead: the dense partial slots.
    Wider layers (three contractions):
    fwdbwd: ids and rows read, W1 read, the per-window vectors (3H floats)
      and the db1/dw2/loss partials written; flops 2HK + 2Hd per window.
    wide_dw1: ids and rows read, the per-window vectors read, one dW1
      partial per 1024-window slice written; flops 2HK + 2Hd per window.
    wide_g: the per-window vectors and W1 read, G written; flops
      (win+1) 2Hd per window.
    sort: 16 B per entry per radix pass (keys and values, read and written).
    update: sorted keys+values and every G row read once, every distinct row
      of E read and written, W1/b1/w2/b2 read and written; flops = one add
      per G element.  Overhead: the dense partials read back.
    segfix: the chunk partials of long rows (d floats each) read, their rows
      read and written.
    """
    d, win, H, K = w.d, w.win, w.H, w.K
    N = B * (win + 1)
    dense = (H * K + 2 * H + 1) * 4
    rows_in = B * ((win + 1) * 4 + (win + 1) * d * 4)
    g_out = B * (win + 1) * d * 4
    if H > 64:
        slices = -(-B // 1024)
        vparts = -(-B // 32)
        vec = B * 3 * H * 4
        part_bytes = slices * H * K * 4 + vparts * (2 * H + 2) * 4
        m = {
            "fwdbwd": (rows_in + H * K * 4 + vec + vparts * (2 * H + 2) * 4,
                       B * (2 * H * K + 2 * H * d), "mfma"),
            "wide_dw1": (rows_in + vec + slices * H * K * 4, B * (2 * H * K + 2 * H * d), "mfma"),
            "wide_g": (vec + H * K * 4 + g_out, B * (win + 1) * 2 * H * d, "mfma"),
        }
    else:
        Hp = _hp(H)
        part_stride = Hp * K + 2 * Hp + 2
        part_bytes = n_parts * part_stride * 4
        m = {
            "fwdbwd": (rows_in + g_out + H * K * 4,
                       B * (4 * H * K + 4 * H * d + (win + 1) * 2 * H * d), "mfma"),
        }
    m["sort"] = (N * 16 * passes, 0, "hbm")
    m["update"] = (N * (8 + d * 4) + 2 * st["U"] * d * 4 + 2 * dense, N * d, "alu")
    m["segfix"] = (st["partials"] * d * 4 + 2 * st["long_rows"] * d * 4, st["partials"] * d, "alu")
    over = {"fwdbwd": part_bytes, "update": part_bytes}
    if H > 64:
        over = {"wide_dw1": slices * H * K * 4, "update": part_bytes}
    return m, over


def roofline(nbytes, nflops, engine, ms):
    """Bound by intensity against the ridge of the kernel's own engine."""
    sec = ms * 1e-3
    peak_f = F32_MATRIX_PEAK_TFLOPS if engine == "mfma" else F32_VECTOR_PEAK_TFLOPS
    ridge = peak_f * 1e12 / (HBM_PEAK_GBS * 1e9)
    if nflops and nbytes and nflops / nbytes > ridge:
        ach = nflops / sec / 1e12
        return {"bound": engine, "achieved": round(ach, 4), "peak": peak_f, "unit": "TFLOP/s",
                "frac": round(ach / peak_f, 5)}
    ach = nbytes / sec / 1e9
    return {"bound": "hbm", "achieved": round(ach, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBS, 5)}


# ---------------------------------------------------------------------------
# HBM traffic from the committed rocprofv3 counter summaries.

def code_text(text):
    """C++ source without comments and without whitespace runs: the part of a
    file that the compiler sees (string literals here contain no comment
    markers)."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_digest(src=None):
    """sha256 over the HIP sources' code (file names and comment-free text,
    sorted by name): a comment edit keeps the counters valid, a code edit
    does not."""
    import hashlib
    h = hashlib.sha256()
    src = src or os.path.join(ROOT, "paper_1404_1521_amd", "csrc")
    for name in sorted(os.listdir(src)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode())
            with open(os.path.join(src, name), encoding="utf-8") as f:
                h.update(code_text(f.read()).encode())
    return h.hexdigest()


def counter_traffic(summary, kernel):
    """HBM bytes per launch (per call for the scatter-add entries) of `kernel`
    from the summary's FETCH_SIZE and WRITE_SIZE averages, each scaled by the
    ratio of known bytes to counted bytes of a plain device copy profiled the
    same way.  None if the summary is missing, lacks the kernel, or was taken
    from kernel sources other than the ones built here."""
    import re
    try:
        with open(COUNTERS.format(summary)) as f:
            text = f.read()
    except OSError:
        return None
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return None
    data = json.loads(m.group(1))
    k = data.get("kernels", {}).get(kernel)
    if data.get("source_sha256") != source_digest() or not k:
        return None
    cal = data["copy"]
    f_scale = cal["bytes_read"] / (cal["fetch_kib"] * 1024.0)
    w_scale = cal["bytes_written"] / (cal["write_kib"] * 1024.0)
    return int(round(k["fetch_kib"] * 1024.0 * f_scale + k["write_kib"] * 1024.0 * w_scale))


def cpu_model_name():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(w, seconds):
    """The float64-arithmetic C++ oracle, one thread, on the first steps of the workload."""
    import oracle
    import workloads
    p = workloads.init_params(w)
    steps, busy = 0, 0.0
    # pinned to one core of those this process may use, for the timed steps
    allowed = sorted(os.sched_getaffinity(0))
    core = allowed[0]
    os.sched_setaffinity(0, {core})
    try:
        while busy < seconds:
            win, cor = workloads.batch(w, steps, w.B)
            a = time.perf_counter()
            oracle.train_step(p, win, cor, w.lr)
            busy += time.perf_counter() - a
            steps += 1
    finally:
        os.sched_setaffinity(0, set(allowed))
    return {
        "value": round(w.B * steps / busy, 1),
        "unit": "windows/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"first {steps} steps of {w.name} (B={w.B}): float32 storage, float64 "
                  f"arithmetic C++ oracle, 1 thread pinned to core {core} ({len(allowed)} cores "
                  f"allowed, {os.cpu_count()} in the machine) on {cpu_model_name()}, "
                  f"{busy:.1f} s of step time",
    }


def time_events(torch, stream, fn, reps):
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    fn()
    stream.synchronize()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    stream.synchronize()
    return e0.elapsed_time(e1) / reps


def kernel_rooflines(torch, np, pg, workloads, stream, reps=20):
    """Standalone gather (B = 16,384 windows over the 1M x 128 stress table,
    and B = 65,536 over the cache-resident 100k x 64 table), scatter-add
    (327,680 Zipf(1.2) rows into a 100k x 64 table) and the general op
    (bfloat16 increment with int64 ids, binary16 assignment with int32 ids,
    same workload) with
    their HBM rooflines.  Durations are the library's per-kernel events (bound
    to the dispatch).  A scatter-add or general-op roofline covers the
    table-update kernels (the sort is reported separately, as its bytes are
    not the operation's); whole calls are timed end to end on the stream as
    well."""
    out = {}
    # The gather, twice: over the stress table (1M x 128 floats, 512 MB,
    # twice the 256 MB Infinity Cache) and over the 100k x 64 table (25.6 MB,
    # cache-resident).  Algorithmic bytes: the ids, every DISTINCT row read
    # once (a repeated row is read from cache, not from HBM) and X and Xc
    # written; the per-window figure that counts every row read is given
    # beside it.
    for key, name in (("gather", "stress"), ("gather_cache_resident", "sweep_65536")):
        w = workloads.PRESETS[name]
        gctx = pg.Context(w.V, w.d, w.win, w.H, max_batch=w.B, stream=stream)
        try:
            p = workloads.init_params(w)
            E = torch.from_numpy(p["E"]).cuda()
            del p
            wins, cors = workloads.batch(w, 0, w.B)
            dw, dc = torch.from_numpy(wins).cuda(), torch.from_numpy(cors).cuda()
            X = torch.empty(w.B, w.K, device="cuda")
            Xc = torch.empty(w.B, w.d, device="cuda")
            gctx.gather(E, dw, dc, X, Xc)
            stream.synchronize()
            gctx.set_timing(True)
            for _ in range(reps):
                gctx.gather(E, dw, dc, X, Xc)
            ms, n = gctx.kernel_times()["gather"]
            if gctx.status() != pg.OK:
                raise RuntimeError("device error flag raised in the gather measurement")
        finally:
            gctx.close()
        U = int(np.unique(np.concatenate([wins.ravel(), cors])).size)
        ids_b = w.B * (w.win + 1) * 4
        out_b = w.B * (w.win + 1) * w.d * 4
        nbytes = ids_b + U * w.d * 4 + out_b
        out[key] = dict(roofline(nbytes, 0, "hbm", ms / n),
                        traffic=counter_traffic("kernels", key),
                        avg_launch_us=round(ms / n * 1e3, 3), bytes_per_launch=nbytes,
                        bytes_per_launch_every_row=ids_b + 2 * out_b, distinct_rows=U,
                        table_mb=round(w.V * w.d * 4 / 1e6, 1),
                        workload=f"B={w.B} V={w.V} d={w.d} win={w.win} Zipf({w.zipf_s})")
        del E, dw, dc, X, Xc
    torch.cuda.empty_cache()

    w = workloads.PRESETS["sweep_65536"]
    sw = workloads.SCATTER_ISO
    ctx = pg.Context(w.V, w.d, w.win, w.H, max_batch=w.B, max_scatter=sw.N, max_rows=sw.rows,
                     stream=stream)
    try:

        table0, idx, Y = workloads.scatter_inputs(sw)
        T = torch.from_numpy(table0).cuda()
        I = torch.from_numpy(idx).cuda()
        Yd = torch.from_numpy(Y).cuda()
        U = int(np.unique(idx).size)
        nbytes = sw.N * (4 + 4 * sw.d) + 2 * U * sw.d * 4
        ctx.set_timing(False)
        for name, mode in (("scatter_sorted", pg.SCATTER_SORTED), ("scatter_atomic", pg.SCATTER_ATOMIC)):
            # whole calls back to back (every launch of the call and the gaps
            # between them), then the same calls with per-kernel events.  The
            # roofline is the table update's kernels (segmented apply + fix-up,
            # or the atomic adds); the sort is reported beside it
            call_ms = time_events(torch, stream, lambda: ctx.scatter_add(T, I, Yd, 1.0, mode), reps)
            ctx.set_timing(True)
            for _ in range(reps):
                ctx.scatter_add(T, I, Yd, 1.0, mode)
            kt = ctx.kernel_times()
            ctx.set_timing(False)
            us = {k: kt[k][0] / reps * 1e3 for k in ("sort", "scatter", "segfix")}
            table_ms = (us["scatter"] + us["segfix"]) * 1e-3
            call = roofline(nbytes, 0, "hbm", call_ms)
            out[name] = dict(roofline(nbytes, 0, "hbm", table_ms), traffic=counter_traffic("kernels", name),
                             table_kernels_us=round(table_ms * 1e3, 3),
                             sort_us_per_call=round(us["sort"], 3),
                             apply_us_per_call=round(us["scatter"], 3),
                             fixup_us_per_call=round(us["segfix"], 3),
                             avg_call_us=round(call_ms * 1e3, 3),
                             call_achieved=call["achieved"], call_frac=call["frac"],
                             launches_per_call=sum(kt[k][1] for k in ("sort", "scatter", "segfix")) // reps,
                             bytes_per_call=nbytes,
                             workload=f"{sw.N} rows Zipf({sw.zipf_s}) into {sw.rows}x{sw.d}, U={U}")
        ctx.set_timing(False)
        # the general op on the same workload: a bfloat16 table with int64
        # indices (increment), and a float16 table (assignment).  Roofline of
        # the table kernels: increment 4 B sorted key + 2d B of Y per entry and
        # 2 * 2d B per distinct row; assignment 8 B (key, entry) per entry and
        # 2 * 2d B per distinct row (one Y row read, one table row written)
        I64 = I.to(torch.int64)
        for name, dt, ix, op, gbytes in (
                ("update_bf16_inc", torch.bfloat16, I64, pg.OP_INC,
                 sw.N * (4 + 2 * sw.d) + 2 * U * sw.d * 2),
                ("update_f16_set", torch.float16, I, pg.OP_SET, sw.N * 8 + 2 * U * sw.d * 2)):
            Tg, Yg = T.to(dt), Yd.to(dt)
            call_ms = time_events(torch, stream, lambda: ctx.scatter_update(Tg, ix, Yg, 1.0, op), reps)
            ctx.set_timing(True)
            for _ in range(reps):
                ctx.scatter_update(Tg, ix, Yg, 1.0, op)
            kt = ctx.kernel_times()
            ctx.set_timing(False)
            us = {k: kt.get(k, (0.0, 0))[0] / reps * 1e3 for k in ("sort", "scatter", "segfix")}
            table_ms = (us["scatter"] + us["segfix"]) * 1e-3
            out[name] = dict(roofline(gbytes, 0, "hbm", table_ms), traffic=counter_traffic("kernels", name),
                             table_kernels_us=round(table_ms * 1e3, 3),
                             sort_us_per_call=round(us["sort"], 3),
                             apply_us_per_call=round(us["scatter"], 3),
                             fixup_us_per_call=round(us["segfix"], 3),
                             avg_call_us=round(call_ms * 1e3, 3), bytes_per_call=gbytes,
                             workload=f"{sw.N} rows Zipf({sw.zipf_s}) into {sw.rows}x{sw.d} {dt}, "
                                      f"{'int64' if ix.dtype == torch.int64 else 'int32'} ids")
        if ctx.status() != pg.OK:
            raise RuntimeError("device error flag raised in the kernel measurements")
    finally:
        ctx.close()
    return out


def convergence_study(torch, np, pg, workloads, budget, target):
    """Batch size against convergence (the paper's §4.6 question, on the
    planted task of workloads.PLANTED): for each batch size and learning-rate
    schedule, train until the held-out ranking error reaches `target` or
    `budget` windows are spent; report windows, steps and GPU seconds (the
    train_steps calls only, between stream synchronisations; data generation
    and evaluation excluded)."""
    task = workloads.PLANTED
    ew, ewc = task.held_out()
    dew, dewc = torch.from_numpy(ew).cuda(), torch.from_numpy(ewc).cuda()
    s_true = torch.empty(ew.shape[0], device="cuda")
    s_cor = torch.empty(ew.shape[0], device="cuda")
    chunk = 65536  # training windows between evaluations
    runs = []
    for sched, lr_of in (("lr 1.0", lambda B: 1.0),
                         ("lr 0.25*sqrt(B/16)", lambda B: 0.25 * (B / 16) ** 0.5)):
        for B in (16, 64, 256, 1024, 4096):
            lr = lr_of(B)
            pd = {k: torch.from_numpy(v).cuda()
                  for k, v in workloads.init_params(task.workload(B, lr)).items()}
            ctx = pg.Context(task.V, task.d, task.win, task.H, max_batch=max(B, ew.shape[0]))
            S = max(1, chunk // B)
            dw = torch.empty(S, B, task.win, dtype=torch.int32, device="cuda")
            dc = torch.empty(S, B, dtype=torch.int32, device="cuda")
            losses = torch.zeros(S, device="cuda")
            rng = np.random.default_rng([task.seed, 4, B])
            seen = steps = 0
            gpu_s, err, curve = 0.0, 1.0, []
            while seen < budget:
                w, c = task.batch(rng, S * B)
                dw.copy_(torch.from_numpy(w.reshape(S, B, task.win)))
                dc.copy_(torch.from_numpy(c.reshape(S, B)))
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                ctx.train_steps(pd, dw, dc, lr, losses)  # same buffers: the cached graph replays
                torch.cuda.synchronize()
                gpu_s += time.perf_counter() - t0
                seen += S * B
                steps += S
                ctx.score(pd, dew, s_true)
                ctx.score(pd, dewc, s_cor)
                err = float((s_true <= s_cor).float().mean())
                curve.append([seen, round(err, 4)])
                if err <= target:
                    break
            if ctx.status() != pg.OK:
                raise RuntimeError("device error flag raised in the convergence study")
            ctx.close()
            runs.append({"schedule": sched, "B": B, "lr": round(lr, 4), "reached": err <= target,
                         "windows": seen, "steps": steps, "gpu_s": round(gpu_s, 4),
                         "final_error": round(err, 4), "final_loss": round(float(losses.mean()), 4),
                         "curve": curve if len(curve) <= 24 else curve[::len(curve) // 24] + [curve[-1]]})
    return {"study": "batch size vs convergence on the planted synthetic task",
            "task": {"V": task.V, "d": task.d, "win": task.win, "H": task.H, "zipf_s": task.zipf_s,
                     "noise": task.noise, "held_out": int(ew.shape[0])},
            "target_error": target, "budget_windows": budget, "eval_every_windows": chunk,
            "runs": runs}


def copy_ceiling(torch, mib=256, reps=10):
    """Streaming-copy ceiling measured on this device: a plain device-to-device
    copy of `mib` MiB, timed with events on the current stream; bytes read +
    bytes written per second, in GB/s."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        dst.copy_(src)
    t1.record()
    t1.synchronize()
    gbs = 2 * n * 4 * reps / (t0.elapsed_time(t1) * 1e-3) / 1e9
    del src, dst
    return round(gbs, 1)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the step has no "
              "multi-GPU path; see the sharding notes in the design document", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    if args.copy_probe:
        n = args.copy_probe * (1 << 20) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4,
                          "copies": 5}), flush=True)
        return

    import paper_1404_1521_amd as pg
    import workloads

    if args.convergence:
        torch.cuda.set_device(0)
        print(json.dumps(convergence_study(torch, np, pg, workloads, args.conv_budget,
                                           args.conv_target)), flush=True)
        return

    if args.only_kernels:
        torch.cuda.set_device(0)
        stream = torch.cuda.Stream()
        with torch.cuda.stream(stream):
            kernel_rooflines(torch, np, pg, workloads, stream)
        torch.cuda.synchronize()
        return

    w = workloads.PRESETS[args.workload]
    if args.batch:
        w = w.with_batch(args.batch)
    B, K, Wm = w.B, args.steps, args.warmup
    N = B * (w.win + 1)
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
        dwin = torch.from_numpy(wins).cuda()
        dcor = torch.from_numpy(cors).cuda()
        losses = torch.zeros(nb, device="cuda")
        ctx = pg.Context(w.V, w.d, w.win, w.H, max_batch=B, scatter_mode=mode, stream=stream)

        def run(lo, hi):
            if args.eager:
                for s in range(lo, hi):
                    ctx.train_step(pd, dwin[s], dcor[s], w.lr, losses[s:s + 1])
            else:
                ctx.train_steps(pd, dwin[lo:hi], dcor[lo:hi], w.lr, losses[lo:hi])

        for s in range(Wm):
            ctx.train_step(pd, dwin[s], dcor[s], w.lr, losses[s:s + 1])
        if not args.eager:
            run(Wm, Wm + K)  # captures the graph of K steps; the timed call replays it
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
        # spread: the same K steps replayed five more times, each timed alone
        # (value above is the first timed replay)
        reps = []
        for _ in range(5):
            e0.record(stream)
            run(Wm, Wm + K)
            e1.record(stream)
            e1.synchronize()
            reps.append(e0.elapsed_time(e1) / K)
        if ctx.status() != pg.OK:
            raise RuntimeError("device error flag raised during the repeats")

        # per-kernel durations: K more steps, one call each, HIP events around
        # every launch on the library stream
        ctx.set_timing(True)
        for s in range(Wm + K, Wm + 2 * K):
            ctx.train_step(pd, dwin[s], dcor[s], w.lr, losses[s:s + 1])
        kt = ctx.kernel_times()
        ctx.set_timing(False)
        lh = losses.cpu().numpy()
        if not np.all(np.isfinite(lh)):
            raise RuntimeError("non-finite loss")
        kern = None if args.no_kernels else kernel_rooflines(torch, np, pg, workloads, stream)
        ctx.close()
        ceiling = copy_ceiling(torch)

    # structure of the timed batches (sampled) for the byte model
    small = N <= 8192 and w.H <= 64
    samp = [batch_structure(wins[s], cors[s], seg_chunk(N)) for s in range(Wm + K, Wm + K + min(K, 8))]
    st = {k: float(np.mean([x[k] for x in samp])) for k in samp[0]}
    key_bits = max(1, int(w.V - 1).bit_length())
    passes = 0 if small else -(-key_bits // 9)
    # dense-partial slots: one per workgroup of the fused kernel (256 at most
    # for the compile-time shapes d 64 / d 16 with window 5, 512 otherwise)
    nt = -(-w.H // 16)
    n_parts = min(-(-B // 16), 256 if (w.d, w.win, nt) in ((64, 5, 2), (16, 5, 1)) else 512)
    model, overhead = step_model(w, B, st, passes, n_parts)
    model_flops = sum(v[1] for v in model.values())
    per = {k: (v[0] / v[1], v[1] / K) for k, v in kt.items() if v[1]}
    step_us = {k: v[0] * v[1] for k, v in per.items()}
    # A large list's sort runs on a second stream beside the contractions it
    # overlaps (fused kernel, or the wide-layer kernels); it is only the
    # step's dominant kernel when it outlasts them
    cand = dict(step_us)
    if "sort" in cand and cand["sort"] <= sum(cand.get(k, 0.0) for k in ("fwdbwd", "wide_dw1", "wide_g")):
        del cand["sort"]
    dom = max(cand, key=cand.get)
    dms = per[dom][0]
    # the model is per step; a kernel id with several launches per step (the
    # sort: histogram + one launch per radix pass) is priced per launch
    nbytes, nflops, engine = model[dom]
    nbytes, nflops = nbytes / per[dom][1], nflops / per[dom][1]
    roof = roofline(nbytes, nflops, engine, dms)
    # the committed counters are per workload at its own batch size
    own = not args.batch or args.batch == workloads.PRESETS[args.workload].B
    roof["traffic"] = counter_traffic(args.workload, dom) if args.mode == "sorted" and own else None
    roof["traffic_unit"] = "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
    roof["kernel"] = dom
    roof["launches_per_step"] = round(per[dom][1], 3)
    roof["avg_launch_us"] = round(dms * 1e3, 3)
    roof["bytes_per_launch"] = int(nbytes)
    roof["flops_per_launch"] = int(nflops)
    roof["intensity_flop_per_byte"] = round(nflops / nbytes, 3) if nbytes else None
    # traffic this implementation adds beyond the method's bytes (not in `achieved`)
    ob = overhead.get(dom, 0) / per[dom][1]
    roof["overhead_bytes_per_launch"] = int(ob)
    roof["overhead_ratio"] = round((nbytes + ob) / nbytes, 4) if nbytes else None
    roof["kernels_us_per_step"] = {k: round(v[0] * v[1] * 1e3, 3) for k, v in per.items()}
    # every contraction of the step over the step time (all kernels, gaps included)
    roof["step_tflops"] = round(model_flops / (ms / K * 1e-3) / 1e12, 3)
    # the HBM denominator measured here, beside the 8 TB/s of the data sheet
    roof["copy_ceiling_gbs"] = ceiling
    roof["frac_of_copy"] = round(roof["achieved"] / ceiling, 5) if roof["unit"] == "GB/s" else None
    # kernel time per step over step time (above 1 when the side-stream sort
    # overlaps the main stream)
    roof["gpu_busy"] = round(sum(step_us.values()) / (ms / K), 3)  # both in ms

    if kern is not None:
        for kr in kern.values():
            if kr.get("unit") == "GB/s":
                kr["frac_of_copy"] = round(kr["achieved"] / ceiling, 5)
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
                               f"scatter={args.mode} {'eager' if args.eager else 'graph'}",
                   "global_batch": B, "parallelism": "single-gpu",
                   "distinct_rows_per_step": round(st["U"], 1)},
        "roofline": roof,
        "repeats": {"n": len(reps), "ms_per_step_mean": round(float(np.mean(reps)), 5),
                    "ms_per_step_std": round(float(np.std(reps, ddof=1)), 5)},
        "wall_s": round(wall, 4),
    }
    if kern is not None:
        out["kernels"] = kern
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
