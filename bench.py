#!/usr/bin/env python3
"""Latency of the two-layer MLP Y = act(X W1) W2 on one MI355X, in each mode.

A step is one ``mlp2_run`` (the whole hot path: GEMM1 + activation + ready
signals + GEMM2) over one batch of synthetic input already resident in HBM.
The headline workload is the largest single-GPU configuration, the 70B gated
MLP (256 x 8192 x 28672, SwiGLU, seed 3).  W warm-up steps, then exactly K
back-to-back steps of the tile-pipelined mode timed between a synchronise on
each side; ``value`` is that block's mean latency per step, which is the
average duration of the pipelined kernel (one launch per step, HIP events on
the stream it is launched on).  Beside it the line carries:

* the sequential mode's latency: the mean of equal blocks timed just before
  and just after the pipelined one; the workqueue mode's; a repeat of the
  pipelined block and the drift between the two;
* cold latencies of both modes (a 1 GiB read evicts the L2s and the 256 MB
  MALL before each timed run, modes interleaved) and the cold roofline
  fraction; both modes timed run by run in alternating order (medians);
* the roofline of the pipelined launch (algorithmic bytes or flops over its
  duration, against the published peak) with the HBM traffic per launch from
  the committed rocprofv3 counter summary of that workload while it matches
  the current kernel sources, and what the GPU attains outside the library
  (a 4 GiB read-only stream, an 8192^3 hipBLASLt GEMM) as context;
* every MLP workload on its own seeded inputs (the seeds of its
  configuration): both modes blocked, interleaved and cold, the workqueue
  and sentinel modes (the paper's scoreboard queue, and its Lamport-style
  synchronisation without fences or flags), eager PyTorch on
  the same inputs (hipBLASLt GEMMs plus an activation kernel), and the same
  roofline object with traffic;
* the paper's micro-batching comparison on one GPU: 8192 x 8192 weights at
  8192 and 16384 rows, chunks of rows in a two-stream stage pipeline captured
  in a HIP graph, chunk sizes swept, beside the one-launch pipelined and
  sequential modes (graph-captured too);
* the fp64 CPU oracle timed on this host (one full evaluation of the
  headline workload when it fits the budget), with the host's CPU count and
  the BLAS thread count;
* with ``--paper-shapes``, the paper's own workload (8192 x 8192 weights,
  no activation, M = 1024 ... 32768) in every mode, beside eager PyTorch;
* with ``--chain``, the GEMM chain (4 layers of 8192 x 8192, GELU between,
  M from ``--chain-rows``) in both modes, beside eager PyTorch.

Only ``--gpus 1`` is supported: the build targets a single GPU.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "2-layer MLP latency µs (pipelined vs sequential) + % HBM BW / MFMA peak"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
# Sources that decide what a planned launch runs (kernels, tiles, orders): the
# committed HBM traffic of a workload is reported only while their hash matches.
KERNEL_SOURCES = [
    "paper_2607_07862_amd/csrc/mlp2_api.cpp",
    "paper_2607_07862_amd/csrc/mlp2_device.hpp",
    "paper_2607_07862_amd/csrc/mlp2_kernels.hip",
    "paper_2607_07862_amd/csrc/mlp2_launch.h",
    "paper_2607_07862_amd/csrc/mlp2_plan_impl.h",
]
FLUSH_BYTES = 1 << 30
SETTLE_MS = 200


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload_key: str):
    """HBM bytes per pipelined launch from the committed counter summary, if it matches these sources."""
    p = os.path.join(ROOT, "profiles", f"traffic_{workload_key}.json")
    if not os.path.exists(p):
        return None
    try:
        with open(p) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    return d.get("hbm_bytes_per_launch")


def bound_of(w) -> str:
    return "mfma" if w.alg_flops() / w.alg_bytes() > BF16_PEAK_TFLOPS / HBM_PEAK_GBS * 1e3 else "hbm"


def roofline(w, us: float, key: str = None) -> dict:
    """The roofline object of one workload's pipelined launch taking `us` µs:
    algorithmic bytes (or flops) per launch over the launch time, against the
    published peak; HBM traffic per launch from the committed counter summary
    of that workload when it matches the current kernel sources (else null)."""
    if bound_of(w) == "hbm":
        achieved = w.alg_bytes() / (us * 1e-6) / 1e9
        r = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    else:
        achieved = w.alg_flops() / (us * 1e-6) / 1e12
        r = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    r["frac"] = round(achieved / r["peak"], 4)
    r["traffic"] = measured_traffic(key) if key else None
    return r


def device_random_inputs(w):
    """Inputs of the workload's shapes and distributions drawn on the device (timing only)."""
    import torch

    gen = torch.Generator(device="cuda")
    gen.manual_seed(1000 + w.seed)
    n1 = 2 if w.gated else 1
    X = torch.randn(w.M, w.H, device="cuda", generator=gen).to(torch.bfloat16)
    W1 = (torch.randn(n1 * w.H, w.F, device="cuda", generator=gen) * w.H ** -0.5).to(torch.bfloat16)
    W2 = (torch.randn(w.F, w.H, device="cuda", generator=gen) * w.F ** -0.5).to(torch.bfloat16)
    return {"X": X, "W1": W1, "W2": W2}


CHAIN_LAYERS, CHAIN_WIDTH, CHAIN_ROWS = 4, 8192, (128, 1024, 4096, 16384)
CHAIN_ROWS_SHORT = (128, 4096)  # the default run's chain leg (--chain: every row count above)


def chain_row(B, M: int, steps: int, iters: int) -> dict:
    """The GEMM chain of CHAIN_LAYERS layers of CHAIN_WIDTH x CHAIN_WIDTH weights
    (GELU between layers) on M rows: both modes (blocks of `steps` runs, and
    `iters` runs per mode timed one by one in alternating order) and eager
    PyTorch (hipBLASLt GEMMs and a GELU kernel per layer) on the same inputs."""
    import torch
    import torch.nn.functional as Fn

    dims = [CHAIN_WIDTH] * (CHAIN_LAYERS + 1)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2000 + M)
    X = torch.randn(M, dims[0], device="cuda", generator=gen).to(torch.bfloat16)
    Ws = [(torch.randn(dims[l], dims[l + 1], device="cuda", generator=gen) * dims[l] ** -0.5).to(torch.bfloat16)
          for l in range(CHAIN_LAYERS)]
    Y = torch.empty(M, dims[-1], dtype=torch.bfloat16, device="cuda")
    plan = B.ChainPlan(M, dims, B.ACT_GELU_TANH)
    modes = (B.MODE_TILE_PIPELINED, B.MODE_SEQUENTIAL)
    for _ in range(5):
        for m in modes:
            plan.run(X, Ws, Y, m)
    torch.cuda.synchronize()

    def timed(fn, n):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(n):
            fn()
        e.record()
        e.synchronize()
        return s.elapsed_time(e) * 1000 / n

    blocks = {m: timed(lambda m=m: plan.run(X, Ws, Y, m), steps) for m in modes}
    one = {m: [] for m in modes}
    for _ in range(iters):
        for m in modes:
            one[m].append(timed(lambda m=m: plan.run(X, Ws, Y, m), 1))
    assert plan.check() == B.OK
    plan.close()

    def eager():
        Z = X
        for l, W in enumerate(Ws):
            Z = Z @ W
            if l < CHAIN_LAYERS - 1:
                Z = Fn.gelu(Z, approximate="tanh")
        return Z

    eager()
    te = timed(eager, steps)
    flops = 2.0 * M * sum(dims[l] * dims[l + 1] for l in range(CHAIN_LAYERS))
    p_us, s_us = blocks[modes[0]], blocks[modes[1]]
    mp, ms = statistics.median(one[modes[0]]), statistics.median(one[modes[1]])
    return {
        "M": M, "layers": CHAIN_LAYERS, "width": CHAIN_WIDTH,
        "pipelined_us": round(p_us, 2), "sequential_us": round(s_us, 2), "gain_pct": round((s_us - p_us) / s_us * 100, 1),
        "interleaved_median_us": {"pipelined": round(mp, 2), "sequential": round(ms, 2),
                                  "gain_pct": round((ms - mp) / ms * 100, 1)},
        "torch_eager_us": round(te, 2),
        "mfma_frac": round(flops / (p_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4),
    }


# Micro-batching legs: rows of the paper's 8192 x 8192 shapes and the chunk sizes swept at each.
MICROBATCH = {"paper_m8192": (1024, 2048, 4096), "paper_m16384": (2048, 4096, 8192)}


def _graph_of(fn):
    """A HIP graph holding whatever `fn(stream)` enqueues, captured on a side stream."""
    import torch

    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(graph, stream=cap):
        fn(cap)
    torch.cuda.synchronize()
    return graph


def _replay_us(graphs: dict, replays: int) -> dict:
    """Median µs per replay of each graph, graphs replayed in alternating order."""
    import torch

    for gr in graphs.values():
        for _ in range(3):
            gr.replay()
    torch.cuda.synchronize()
    times = {k: [] for k in graphs}
    for _ in range(replays):
        for k, gr in graphs.items():
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            gr.replay()
            b.record()
            b.synchronize()
            times[k].append(a.elapsed_time(b) * 1e3)
    return {k: statistics.median(v) for k, v in times.items()}


def microbatch_row(B, I, key: str, chunks, replays: int) -> dict:
    """The paper's headline comparison (Sec. IV-A: micro-batched execution,
    the chunk size swept and the best kept, the baseline captured in a graph)
    on one GPU.  The rows are cut into chunks of c rows, one plan per chunk;
    chunk i's GEMM1 (the STAGE1 launch) runs on one stream while chunk i-1's
    GEMM2 (STAGE2) runs on a second stream of the same priority, each GEMM2
    ordered after its chunk's GEMM1 by an event, and the whole sequence is
    captured in a HIP graph.  Beside it, one launch over all rows in the
    pipelined and in the sequential mode, each also graph-captured; every
    graph is replayed in alternating order, medians of `replays` replays.
    Inputs are drawn on the device (timing does not depend on the values);
    the micro-batched Y is checked against the one-launch sequential Y."""
    import torch

    w = I.WORKLOADS[key]
    g = device_random_inputs(w)
    X, W1, W2 = g["X"], g["W1"], g["W2"]
    plans, graphs, outs = [], {}, {}

    def whole(mode):
        plan = B.Plan(w.M, w.H, w.F, w.act)
        plans.append(plan)
        Y = torch.empty(w.M, w.H, dtype=torch.bfloat16, device="cuda")
        outs[mode] = Y
        return _graph_of(lambda s: plan.run(X, W1, W2, Y, mode, stream=s))

    graphs["pipelined"] = whole(B.MODE_TILE_PIPELINED)
    graphs["sequential"] = whole(B.MODE_SEQUENTIAL)
    for c in chunks:
        if w.M % c or c >= w.M:
            continue
        cp = [B.Plan(c, w.H, w.F, w.act) for _ in range(w.M // c)]
        plans.extend(cp)
        Y = torch.empty(w.M, w.H, dtype=torch.bfloat16, device="cuda")
        outs[c] = Y

        def chunked(s, cp=cp, Y=Y, c=c):
            s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
            s1.wait_stream(s)
            s2.wait_stream(s)
            for i, plan in enumerate(cp):
                r = slice(i * c, (i + 1) * c)
                plan.run(X[r], W1, W2, Y[r], B.MODE_STAGE1, stream=s1)
                ev = torch.cuda.Event()
                ev.record(s1)
                s2.wait_event(ev)
                plan.run(X[r], W1, W2, Y[r], B.MODE_STAGE2, stream=s2)
            s.wait_stream(s1)
            s.wait_stream(s2)

        graphs[f"microbatch_{c}"] = _graph_of(chunked)
    t = _replay_us(graphs, replays)
    for plan in plans:
        assert plan.check() == B.OK
        plan.close()
    ref = outs[B.MODE_SEQUENTIAL].float()
    scale = ref.abs().max().item()
    row = {"M": w.M, "how": "graph replays, alternating order, medians; micro-batches: STAGE1 and STAGE2 of chunk "
                            "plans on two streams ordered by events"}
    row.update({k: round(v, 2) for k, v in t.items()})
    errs = {}
    for c in chunks:
        if c in outs:
            errs[str(c)] = round((outs[c].float() - ref).abs().max().item() / scale, 6)
    row["microbatch_max_rel_diff_vs_sequential"] = errs
    micro = min((v, k) for k, v in t.items() if k.startswith("microbatch_"))
    row["best_microbatch"] = micro[1]
    row["pipelined_gain_vs_best_microbatch_pct"] = round((micro[0] - t["pipelined"]) / micro[0] * 100, 1)
    row["pipelined_gain_vs_sequential_pct"] = round((t["sequential"] - t["pipelined"]) / t["sequential"] * 100, 1)
    del g, X, W1, W2, outs
    return row


def torch_eager_us(w, g, steps):
    """Mean µs per step of the same MLP in eager PyTorch on the platform
    libraries (hipBLASLt GEMMs plus an elementwise activation kernel), bf16
    in and out, on the same device inputs: a reference point, not the target.
    The gated GEMM1 runs as one GEMM over the gate and up columns side by side."""
    import torch
    import torch.nn.functional as Fn

    X, W2 = g["X"], g["W2"]
    if w.gated:
        W1v = g["W1"].reshape(2, w.H, w.F)
        W1 = torch.cat([W1v[0], W1v[1]], dim=1)  # [H, 2F]: gate columns, then up columns

        def step():
            gu = X @ W1
            return (Fn.silu(gu[:, : w.F]) * gu[:, w.F :]) @ W2
    else:
        W1 = g["W1"]
        gelu = w.act == 1

        def step():
            z = X @ W1
            return (Fn.gelu(z, approximate="tanh") if gelu else z) @ W2

    for _ in range(3):
        step()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) * 1e3 / steps


class Runner:
    def __init__(self, B, w, g, tuning, stream):
        import torch

        self.B, self.w, self.g, self.stream = B, w, g, stream
        self.Y = torch.empty(w.M, w.H, dtype=torch.bfloat16, device="cuda")
        self.plan = B.Plan(w.M, w.H, w.F, w.act, tuning)
        self.info = self.plan.info()

    def run(self, mode):
        self.plan.run(self.g["X"], self.g["W1"], self.g["W2"], self.Y, mode, stream=self.stream)

    def block(self, mode, steps):
        """Mean µs per step of `steps` back-to-back runs (HIP events on the launch stream)."""
        import torch

        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(self.stream)
        for _ in range(steps):
            self.run(mode)
        stop.record(self.stream)
        torch.cuda.synchronize()
        return start.elapsed_time(stop) * 1e3 / steps

    def cold(self, modes, iters, flush):
        """Per-run µs with the caches flushed before every run, modes interleaved.

        The flush reads 1 GiB (a max-reduction into one value): that evicts the
        L2s and the 256 MB last-level cache without leaving dirty lines behind.
        A flush by writing would charge the write-back of its own dirty lines to
        the timed run (measured: a 256 MB stream right after a 1 GiB write reads
        at less than half its bandwidth)."""
        import torch

        sink = torch.empty((), dtype=flush.dtype, device=flush.device)
        out = {m: [] for m in modes}
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters * len(modes))]
        i = 0
        for _ in range(iters):
            for m in modes:
                torch.amax(flush, dim=0, out=sink)
                a, b = evs[i]
                a.record(self.stream)
                self.run(m)
                b.record(self.stream)
                out[m].append((a, b))
                i += 1
        torch.cuda.synchronize()
        return {m: [a.elapsed_time(b) * 1e3 for a, b in v] for m, v in out.items()}

    def interleaved(self, iters, modes=None):
        """Per-run µs of the modes (default: pipelined and sequential), run by
        run in alternating order (ABBA...), warm.

        Clock and thermal drift then reach every mode alike, which back-to-back
        blocks of one mode do not guarantee."""
        import torch

        order = tuple(modes or (self.B.MODE_TILE_PIPELINED, self.B.MODE_SEQUENTIAL))
        out = {m: [] for m in order}
        for i in range(iters):
            for m in (order if i % 2 == 0 else order[::-1]):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(self.stream)
                self.run(m)
                b.record(self.stream)
                out[m].append((a, b))
        torch.cuda.synchronize()
        return {m: [a.elapsed_time(b) * 1e3 for a, b in v] for m, v in out.items()}

    def check(self):
        if self.plan.check() != self.B.OK:
            raise RuntimeError(f"{self.w.name}: a device flag wait timed out")

    def close(self):
        self.plan.close()


def pct(v, q):
    v = sorted(v)
    return v[min(len(v) - 1, max(0, int(round(q * (len(v) - 1)))))]


def attainable():
    """What this GPU reaches outside the library, as context for the roofline
    fractions (which stay against the published peaks): a read-only stream of
    4 GiB (row maxima of a [65536, 16384] fp32 view, far beyond the 256 MB
    last-level cache; a single full reduction reads at little more than half
    that rate) and an 8192^3 bf16 GEMM through torch.matmul (hipBLASLt).
    Best of 5 runs each."""
    import torch

    buf = torch.ones(65536, 16384, dtype=torch.float32, device="cuda")
    sink = torch.empty(65536, dtype=torch.float32, device="cuda")
    a = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    b = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    c = torch.empty(8192, 8192, dtype=torch.bfloat16, device="cuda")

    def best(f, n=5):
        f()
        torch.cuda.synchronize()
        ts = []
        for _ in range(n):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            f()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return min(ts)

    t_read = best(lambda: torch.amax(buf, dim=1, out=sink))
    t_gemm = best(lambda: torch.matmul(a, b, out=c))
    out = {
        "hbm_read_GBs": round(buf.numel() * 4 / t_read / 1e9, 1),
        "bf16_gemm_TFLOPs": round(2 * 8192 ** 3 / t_gemm / 1e12, 1),
        "how": "4 GiB read-only stream (row maxima, torch.amax) and an 8192^3 bf16 torch.matmul (hipBLASLt), best of 5",
    }
    del buf, a, b, c
    torch.cuda.empty_cache()
    return out


def host_cpu_model() -> str:
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, d, budget_s: float):
    """The oracle as it stands, timed on this host: one full evaluation of the
    workload (every output row, the weights decoded once inside the call) when
    a first 32-row call predicts it fits the budget, else as many 32-row calls
    as fit (each decodes the weights again) scaled to all rows."""
    import numpy as np

    from oracle import mlp2_oracle as O
    from paper_2607_07862_amd import inputs as I

    try:
        from threadpoolctl import threadpool_info

        blas = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] + [1])
    except Exception:  # pragma: no cover
        blas = None
    X, W1, W2 = I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"])
    rows_per = min(w.M, 32)
    t0 = time.perf_counter()
    O.mlp2(X, W1, W2, w.M, w.H, w.F, w.act, rows=np.arange(rows_per))
    t_first = time.perf_counter() - t0
    host = {"cpu_count": os.cpu_count(), "blas_threads": blas, "cpu_model": host_cpu_model()}
    if t_first * max(1.0, w.M / rows_per) <= budget_s or w.M <= rows_per:
        t0 = time.perf_counter()
        O.mlp2(X, W1, W2, w.M, w.H, w.F, w.act)
        t_full = time.perf_counter() - t0
        return {"value": round(t_full * 1e6, 1), "unit": "us", "cores": int(blas or os.cpu_count() or 1),
                "kind": "oracle", **host,
                "sample": f"one full evaluation of {w.name} ({w.M} rows; fp64 numpy, weights decoded once in the call)"}
    times, rows_done = [t_first], rows_per
    t_all = time.perf_counter()
    while time.perf_counter() - t_all < budget_s and rows_done < w.M:
        rows = np.arange(rows_done, min(w.M, rows_done + rows_per))
        t0 = time.perf_counter()
        O.mlp2(X, W1, W2, w.M, w.H, w.F, w.act, rows=rows)
        times.append(time.perf_counter() - t0)
        rows_done += len(rows)
    return {"value": round(sum(times) / rows_done * w.M * 1e6, 1), "unit": "us",
            "cores": int(blas or os.cpu_count() or 1), "kind": "oracle", **host,
            "sample": f"{rows_done} output rows of {w.name} in {len(times)} calls of up to {rows_per} rows (fp64 "
                      f"numpy, weights decoded per call), scaled to M={w.M}"}


def table_row(B, I, key: str, stream, steps: int, iters: int, cold_iters: int, flush, tuning=None) -> dict:
    """One workload on its seeded inputs: both modes and the workqueue mode
    (blocks of `steps` runs), both modes run by run in alternating order
    (`iters` each, medians), cold medians (`cold_iters` each, a 1 GiB read
    before every run), eager PyTorch on the same inputs, and the roofline of
    the pipelined launch with its counter-measured HBM traffic."""
    import torch

    wk = I.WORKLOADS[key]
    gk = {k: v.to("cuda") for k, v in I.workload_inputs(wk).items()}
    rr = Runner(B, wk, gk, tuning, stream)
    for _ in range(20):
        rr.run(B.MODE_TILE_PIPELINED)
        rr.run(B.MODE_SEQUENTIAL)
        rr.run(B.MODE_WORKQUEUE)
        rr.run(B.MODE_SENTINEL)
    s_before = rr.block(B.MODE_SEQUENTIAL, steps)
    p_us = rr.block(B.MODE_TILE_PIPELINED, steps)
    s_us = (s_before + rr.block(B.MODE_SEQUENTIAL, steps)) / 2
    q_us = rr.block(B.MODE_WORKQUEUE, steps)
    n_us = rr.block(B.MODE_SENTINEL, steps)
    ivk = rr.interleaved(iters, (B.MODE_TILE_PIPELINED, B.MODE_SEQUENTIAL, B.MODE_SENTINEL))
    mp, ms = statistics.median(ivk[B.MODE_TILE_PIPELINED]), statistics.median(ivk[B.MODE_SEQUENTIAL])
    mn = statistics.median(ivk[B.MODE_SENTINEL])
    cold = rr.cold([B.MODE_TILE_PIPELINED, B.MODE_SEQUENTIAL], cold_iters, flush) if cold_iters else None
    rr.check()
    inf = rr.info
    rr.close()
    te = torch_eager_us(wk, gk, steps)
    del gk
    torch.cuda.empty_cache()
    rf = roofline(wk, p_us, key)
    row = {
        "pipelined_us": round(p_us, 2),
        "sequential_us": round(s_us, 2),
        "gain_pct": round((s_us - p_us) / s_us * 100, 1),
        "workqueue_us": round(q_us, 2),
        "sentinel_us": round(n_us, 2),
        "interleaved_median_us": {"pipelined": round(mp, 2), "sequential": round(ms, 2), "sentinel": round(mn, 2),
                                  "gain_pct": round((ms - mp) / ms * 100, 1)},
        "torch_eager_us": round(te, 2),
        "roofline": rf,
        "hbm_frac": round(wk.alg_bytes() / (p_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        "mfma_frac": round(wk.alg_flops() / (p_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4),
        "tiles": {k: inf[k] for k in ("bm", "bn1", "splitk1", "bn2", "splitk2", "stages", "waves", "grid_pipelined",
                                      "lag")},
        "seed": wk.seed,
    }
    if cold:
        cp, cs = statistics.median(cold[B.MODE_TILE_PIPELINED]), statistics.median(cold[B.MODE_SEQUENTIAL])
        row["cold_median_us"] = {"pipelined": round(cp, 2), "sequential": round(cs, 2),
                                 "gain_pct": round((cs - cp) / cs * 100, 1)}
        row["cold_roofline_frac"] = roofline(wk, cp)["frac"]
    return row


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20, help="untimed warm-up steps of the headline (each mode once per step)")
    ap.add_argument("--workload", default="l70b_gated",
                    help="headline workload (default: the largest single-GPU configuration, the 70B gated MLP)")
    ap.add_argument("--tuning", default="", help="JSON dict of mlp2_tuning_t fields")
    ap.add_argument("--cpu-budget", type=float, default=60.0,
                    help="longest the CPU oracle may take; beyond it a row sample is timed and scaled")
    ap.add_argument("--cold-iters", type=int, default=20)
    ap.add_argument("--interleave-iters", type=int, default=100,
                    help="warm runs per mode timed one by one in alternating order (0 skips; half of it per table row)")
    ap.add_argument("--no-attainable", action="store_true", help="skip the stream and library-GEMM references")
    ap.add_argument("--no-microbatch", action="store_true",
                    help="skip the micro-batching comparison (8192 x 8192 weights at 8192 and 16384 rows)")
    ap.add_argument("--microbatch-replays", type=int, default=10)
    ap.add_argument("--chain", action="store_true",
                    help="time the GEMM chain (4 layers of 8192 x 8192 weights, GELU between) at every row count "
                         "(the default run times it at 128 and 4096 rows)")
    ap.add_argument("--no-chain", action="store_true", help="skip the GEMM chain leg")
    ap.add_argument("--chain-rows", default="",
                    help="row counts of the chain leg (comma-separated; default 128,1024,4096,16384 with --chain)")
    ap.add_argument("--paper-shapes", action="store_true",
                    help="also time the paper's own workload: 8192x8192 weights, no activation, M = 1024 ... 32768")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle timing")
    ap.add_argument("--no-table", action="store_true", help="skip the table of all workloads")
    ap.add_argument("--only-pipelined", action="store_true", help="time the pipelined mode only (profiling runs)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="first copy MIB MiB device-to-device (a plain copy kernel of known size, for counter scaling)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library runs the hot path on a single MI355X (use --gpus 1)",
              file=sys.stderr)
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

    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: 3 copies of {args.copy_calibration} MiB")
        del src, dst

    # ---- headline workload: the seeded inputs
    w = I.WORKLOADS[args.workload]
    log(f"workload {w.name}: generating seeded inputs (seed {w.seed})")
    d = I.workload_inputs(w)
    g = {k: v.to("cuda") for k, v in d.items()}
    r = Runner(B, w, g, tuning, stream)
    log(f"plan {r.info}")
    # Clock settling: the chip raises its clocks over the first tens of
    # milliseconds of load, so the modes run untimed for SETTLE_MS first (a
    # first timed block otherwise reads a few percent slow); then the
    # warm-up steps.
    t_settle = time.perf_counter()
    while (time.perf_counter() - t_settle) * 1e3 < SETTLE_MS:
        for _ in range(5):
            r.run(B.MODE_TILE_PIPELINED)
            if not args.only_pipelined:
                r.run(B.MODE_SEQUENTIAL)
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        r.run(B.MODE_TILE_PIPELINED)
        if not args.only_pipelined:
            r.run(B.MODE_SEQUENTIAL)
            r.run(B.MODE_WORKQUEUE)
    torch.cuda.synchronize()
    r.check()
    seq_before = None if args.only_pipelined else r.block(B.MODE_SEQUENTIAL, args.steps)
    log(f"timing {args.steps} pipelined steps")
    value = r.block(B.MODE_TILE_PIPELINED, args.steps)
    extra = {}
    flush = None
    if not args.only_pipelined:
        # sequential blocks on both sides of the pipelined one: a drift of the
        # clocks over the blocks reaches the two modes alike
        seq_after = r.block(B.MODE_SEQUENTIAL, args.steps)
        seq_us = (seq_before + seq_after) / 2
        wq_us = r.block(B.MODE_WORKQUEUE, args.steps)
        pipe2 = r.block(B.MODE_TILE_PIPELINED, args.steps)
        log(f"pipelined {value:.2f} us (repeat {pipe2:.2f}), sequential {seq_us:.2f} us, workqueue {wq_us:.2f} us")
        extra = {
            "sequential_us": round(seq_us, 3),
            "sequential_before_after_us": [round(seq_before, 3), round(seq_after, 3)],
            "workqueue_us": round(wq_us, 3),
            "pipelined_repeat_us": round(pipe2, 3),
            "drift_pct": round((pipe2 - value) / value * 100, 2),
            "gain_vs_sequential_pct": round((seq_us - value) / seq_us * 100, 2),
        }
        flush = torch.ones(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
        if args.cold_iters > 0:
            cold = r.cold([B.MODE_TILE_PIPELINED, B.MODE_SEQUENTIAL], args.cold_iters, flush)
            cp, cs = cold[B.MODE_TILE_PIPELINED], cold[B.MODE_SEQUENTIAL]
            extra["cold"] = {
                "pipelined_median_us": round(statistics.median(cp), 2),
                "pipelined_p10_p90_us": [round(pct(cp, 0.1), 2), round(pct(cp, 0.9), 2)],
                "sequential_median_us": round(statistics.median(cs), 2),
                "sequential_p10_p90_us": [round(pct(cs, 0.1), 2), round(pct(cs, 0.9), 2)],
                "roofline_frac": roofline(w, statistics.median(cp))["frac"],
                "iters": args.cold_iters,
                "flush": "1 GiB device read before each timed run (evicts L2 and the last-level cache), modes interleaved",
            }
            log(f"cold: pipelined {extra['cold']['pipelined_median_us']} us, sequential {extra['cold']['sequential_median_us']} us")
        if args.interleave_iters > 0:
            iv = r.interleaved(args.interleave_iters)
            ip, is_ = iv[B.MODE_TILE_PIPELINED], iv[B.MODE_SEQUENTIAL]
            mp, ms = statistics.median(ip), statistics.median(is_)
            extra["interleaved"] = {
                "pipelined_median_us": round(mp, 2),
                "pipelined_p10_p90_us": [round(pct(ip, 0.1), 2), round(pct(ip, 0.9), 2)],
                "sequential_median_us": round(ms, 2),
                "sequential_p10_p90_us": [round(pct(is_, 0.1), 2), round(pct(is_, 0.9), 2)],
                "gain_median_pct": round((ms - mp) / ms * 100, 2),
                "iters": args.interleave_iters,
                "how": "warm, one HIP event pair per run, modes alternating run by run",
            }
            log(f"interleaved: pipelined {mp:.2f} us, sequential {ms:.2f} us")
    r.check()
    info = r.info
    roof = roofline(w, value, args.workload)
    roof["kernel"] = "k_mlp2 pipelined launch (one per step)"
    r.close()
    del g
    torch.cuda.empty_cache()

    # ---- every workload on its seeded inputs
    table = {}
    if not args.no_table and not args.only_pipelined:
        for key in I.WORKLOAD_ORDER:
            row = table_row(B, I, key, stream, max(10, args.steps), max(10, args.interleave_iters // 2),
                            max(0, args.cold_iters // 2), flush)
            table[key] = row
            log(f"TABLE {key:12s} {row}")

    microbatch = {}
    if not args.no_microbatch and not args.only_pipelined:
        for key, chunks in MICROBATCH.items():
            microbatch[key] = microbatch_row(B, I, key, chunks, args.microbatch_replays)
            log(f"MICROBATCH {key:14s} {microbatch[key]}")
            torch.cuda.empty_cache()

    chain = {}
    # the chain leg: every row count with --chain, a short one in the full default run
    if args.chain or (not args.no_chain and not args.no_table and not args.only_pipelined):
        rows = args.chain_rows or ",".join(str(m) for m in (CHAIN_ROWS if args.chain else CHAIN_ROWS_SHORT))
        for Mc in [int(x) for x in rows.split(",")]:
            row = chain_row(B, Mc, max(5, args.steps // 5), 10)
            chain[f"chain{CHAIN_LAYERS}x{CHAIN_WIDTH}_m{Mc}"] = row
            log(f"CHAIN m{Mc:<6d} {row}")
            torch.cuda.empty_cache()

    paper = {}
    if args.paper_shapes:
        for key in I.PAPER_ORDER:
            wk = I.WORKLOADS[key]
            gk = device_random_inputs(wk)
            rr = Runner(B, wk, gk, None, stream)
            for _ in range(5):
                rr.run(B.MODE_TILE_PIPELINED)
                rr.run(B.MODE_SEQUENTIAL)
                rr.run(B.MODE_WORKQUEUE)
            steps = max(5, args.steps // 5)
            s_before = rr.block(B.MODE_SEQUENTIAL, steps)
            p_us = rr.block(B.MODE_TILE_PIPELINED, steps)
            s_us = (s_before + rr.block(B.MODE_SEQUENTIAL, steps)) / 2
            q_us = rr.block(B.MODE_WORKQUEUE, steps)
            ivk = rr.interleaved(10)
            rr.check()
            inf = rr.info
            rr.close()
            te = torch_eager_us(wk, gk, steps)
            del gk
            torch.cuda.empty_cache()
            mp, ms = statistics.median(ivk[B.MODE_TILE_PIPELINED]), statistics.median(ivk[B.MODE_SEQUENTIAL])
            row = {
                "M": wk.M, "pipelined_us": round(p_us, 2), "sequential_us": round(s_us, 2),
                "gain_pct": round((s_us - p_us) / s_us * 100, 1), "workqueue_us": round(q_us, 2),
                "interleaved_median_us": {"pipelined": round(mp, 2), "sequential": round(ms, 2),
                                          "gain_pct": round((ms - mp) / ms * 100, 1)},
                "torch_eager_us": round(te, 2),
                "mfma_frac": round(wk.alg_flops() / (p_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4),
                "tiles": [inf["bm"], inf["bn1"], inf["splitk1"], inf["bn2"], inf["splitk2"], inf["stages"],
                          inf["waves"]],
            }
            paper[key] = row
            log(f"PAPER {key:14s} {row}")
    del flush
    torch.cuda.empty_cache()

    att = None
    if not args.no_attainable:
        att = attainable()
        log(f"attainable: {att}")
        roof["frac_of_attainable"] = round(
            roof["achieved"] / (att["hbm_read_GBs"] if roof["bound"] == "hbm" else att["bf16_gemm_TFLOPs"]), 4)
        for key, row in table.items():
            rf = row["roofline"]
            rf["frac_of_attainable"] = round(
                rf["achieved"] / (att["hbm_read_GBs"] if rf["bound"] == "hbm" else att["bf16_gemm_TFLOPs"]), 4)

    cpu = None
    if not args.no_cpu:
        log(f"timing the CPU oracle (budget {args.cpu_budget}s)")
        cpu = cpu_baseline(w, d, args.cpu_budget)
        log(f"cpu baseline: {cpu}")
        # the oracle on every table row's own seeded inputs (the headline's row: the timing above)
        for key, row in table.items():
            o = cpu if key == args.workload else cpu_baseline(I.WORKLOADS[key], I.workload_inputs(I.WORKLOADS[key]),
                                                              args.cpu_budget)
            row["cpu_oracle"] = {k: o[k] for k in ("value", "unit", "sample")}
            log(f"cpu oracle {key:12s} {row['cpu_oracle']}")

    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "clock_settle_ms": SETTLE_MS,
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
            "seed": w.seed,
            "mode": "tile_pipelined",
            "tiles": {k: info[k] for k in ("bm", "bn1", "splitk1", "bn2", "splitk2", "stages", "waves", "items1",
                                           "items2", "grid_pipelined", "occupancy", "lag")},
        },
        **extra,
        "alg_bytes": w.alg_bytes(),
        "alg_flops": w.alg_flops(),
        "roofline": roof,
        "attainable": att,
        "cpu_baseline": cpu,
        "workloads": table,
        **({"microbatch": microbatch} if microbatch else {}),
        **({"paper_shapes": paper} if paper else {}),
        **({"chain": chain} if chain else {}),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
