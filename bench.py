#!/usr/bin/env python3
"""Latency of the two-layer MLP Y = act(X W1) W2 on one MI355X, both modes.

A step is one ``mlp2_run`` (the whole hot path: GEMM1 + activation + ready
signals + GEMM2) over one batch of synthetic inputs already resident in HBM.
W warm-up steps, then exactly K back-to-back steps of the tile-pipelined mode
timed between a synchronise on each side, then the same for the sequential
mode.  The JSON line on stdout carries the pipelined latency as ``value``,
the sequential latency beside it, the roofline fraction of the dominant
kernel (HIP events on the launch stream) and the CPU oracle timed on a
bounded sample.

Only ``--gpus 1`` is supported: the build targets a single GPU.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "2-layer MLP latency µs (pipelined vs sequential) + % HBM BW / MFMA peak"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
KERNEL_SOURCES = ["paper_2607_07862_amd/csrc/mlp2_device.hpp", "paper_2607_07862_amd/csrc/mlp2_kernels.hip"]


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload_key: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, if it matches these sources."""
    p = os.path.join(ROOT, "profiles", f"traffic_{workload_key}.json")
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
    except Exception:
        return None
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    return d.get("bytes_per_launch")


def time_block(plan, g, Y, mode, steps, stream):
    import torch

    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(steps):
        plan.run(g["X"], g["W1"], g["W2"], Y, mode, stream=stream)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return start.elapsed_time(stop) * 1e3 / steps, wall  # us per step (events), wall seconds


def cpu_baseline(w, d, budget_s: float):
    """The oracle as it stands, timed on this host on a bounded sample of the workload."""
    import numpy as np

    from oracle import mlp2_oracle as O
    from paper_2607_07862_amd import inputs as I

    try:
        from threadpoolctl import threadpool_info

        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    X, W1, W2 = I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"])
    # Sample: row blocks of the workload, as many as fit the time budget
    # (each evaluation decodes the weights and runs both fp64 GEMMs).
    rows_per = min(w.M, 32)
    times, rows_done = [], 0
    t_all = time.perf_counter()
    while True:
        rows = np.arange(rows_done % w.M, rows_done % w.M + rows_per) % w.M
        t0 = time.perf_counter()
        O.mlp2(X, W1, W2, w.M, w.H, w.F, w.act, rows=rows)
        times.append(time.perf_counter() - t0)
        rows_done += rows_per
        if time.perf_counter() - t_all > budget_s or rows_done >= 4 * w.M:
            break
    per_row = sum(times) / rows_done
    return {
        "value": per_row * w.M * 1e6,
        "unit": "us",
        "cores": int(cores),
        "kind": "oracle",
        "sample": f"{rows_done} output rows in {len(times)} calls of {rows_per} rows (fp64 numpy, weights decoded per "
        f"call); value = measured time per row x M={w.M}",
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="l8b_decode")
    ap.add_argument("--tuning", default="", help="JSON dict of mlp2_tuning_t fields")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--all", action="store_true", help="also time every workload (stderr table)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build runs on a single MI355X (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_07862_amd import binding as B
    from paper_2607_07862_amd import inputs as I

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    B.load()  # fails loudly without the compiled library
    stream = torch.cuda.current_stream()
    tuning = json.loads(args.tuning) if args.tuning else None

    def bench_workload(key, steps, warmup):
        w = I.WORKLOADS[key]
        log(f"workload {w.name}: generating inputs (seed {w.seed})")
        d = I.workload_inputs(w)
        g = {k: v.to("cuda") for k, v in d.items()}
        Y = torch.empty(w.M, w.H, dtype=torch.bfloat16, device="cuda")
        plan = B.Plan(w.M, w.H, w.F, w.act, tuning)
        info = plan.info()
        for _ in range(warmup):
            plan.run(g["X"], g["W1"], g["W2"], Y, B.MODE_TILE_PIPELINED, stream=stream)
            plan.run(g["X"], g["W1"], g["W2"], Y, B.MODE_SEQUENTIAL, stream=stream)
        torch.cuda.synchronize()
        if plan.check() != B.OK:
            raise RuntimeError("device flag wait timed out during warm-up")
        pipe_us, wall = time_block(plan, g, Y, B.MODE_TILE_PIPELINED, steps, stream)
        seq_us, _ = time_block(plan, g, Y, B.MODE_SEQUENTIAL, steps, stream)
        pipe_us2, _ = time_block(plan, g, Y, B.MODE_TILE_PIPELINED, steps, stream)
        if plan.check() != B.OK:
            raise RuntimeError("device flag wait timed out during timing")
        log(f"{w.name}: pipelined {pipe_us:.2f} / {pipe_us2:.2f} us, sequential {seq_us:.2f} us  info={info}")
        return w, d, plan, info, pipe_us, seq_us, pipe_us2, wall

    if args.all:
        for key in I.WORKLOAD_ORDER:
            if key == args.workload:
                continue
            w, _, plan, info, p, s, p2, _ = bench_workload(key, max(10, args.steps // 2), 3)
            bound = "mfma" if w.alg_flops() / w.alg_bytes() > BF16_PEAK_TFLOPS / HBM_PEAK_GBS * 1e3 else "hbm"
            pm = min(p, p2)
            log(f"TABLE {key} pipelined_us={pm:.2f} sequential_us={s:.2f} gain={(s - pm) / s * 100:.1f}% "
                f"hbm={w.alg_bytes() / pm / 1e3:.0f}GB/s ({w.alg_bytes() / pm / 1e3 / HBM_PEAK_GBS * 100:.1f}%) "
                f"mfma={w.alg_flops() / pm / 1e6:.0f}TF/s ({w.alg_flops() / pm / 1e6 / BF16_PEAK_TFLOPS * 100:.1f}%) "
                f"bound={bound}")
            plan.close()
            torch.cuda.empty_cache()

    w, d, plan, info, pipe_us, seq_us, pipe_us2, wall = bench_workload(args.workload, args.steps, args.warmup)
    value = pipe_us  # the first timed block of exactly K pipelined steps
    bound = "mfma" if w.alg_flops() / w.alg_bytes() > BF16_PEAK_TFLOPS / HBM_PEAK_GBS * 1e3 else "hbm"
    if bound == "hbm":
        achieved = w.alg_bytes() / (value * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    else:
        achieved = w.alg_flops() / (value * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    roof["frac"] = round(achieved / roof["peak"], 4)
    roof["traffic"] = measured_traffic(args.workload)
    roof["kernel"] = "k_pipelined (one launch per step)"

    cpu = None
    if not args.no_cpu:
        log(f"timing the CPU oracle (budget {args.cpu_budget}s)")
        cpu = cpu_baseline(w, d, args.cpu_budget)

    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(value / 1e3, 6),
        "higher_is_better": False,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "M": w.M,
            "H": w.H,
            "F": w.F,
            "act": ["identity", "gelu_tanh", "swiglu"][w.act],
            "mode": "tile_pipelined",
            "tiles": {k: info[k] for k in ("bm", "bn1", "splitk1", "bn2", "splitk2", "items1", "items2",
                                           "grid_pipelined", "occupancy")},
        },
        "sequential_us": round(seq_us, 3),
        "pipelined_repeat_us": round(pipe_us2, 3),
        "gain_vs_sequential_pct": round((seq_us - value) / seq_us * 100, 2),
        "alg_bytes": w.alg_bytes(),
        "alg_flops": w.alg_flops(),
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    plan.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
