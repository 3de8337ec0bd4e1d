"""Where the time of one run goes, from the per-item timing trace.

    python -m paper_2607_07862_amd.tracesum [--workloads a,b,...] [--out FILE.md]

Needs the trace build (``python -m paper_2607_07862_amd.build --trace``) and
a GPU.  For each workload (device-drawn inputs of its shapes): warm-up runs,
then one traced warm run per mode.  Per item kind it reports the mean item
time split into mainloop, waits for the work-group's own ring loads, flag
waits (ready counters in the pipelined mode; re-reads of intermediate pieces
still holding the sentinel in the sentinel mode; in the workqueue mode the wait
for the popped queue slot to fill, counted from when the work-group began to
pop) and epilogue, the item's core clock cycles and the clock they imply
(cycles over real time), and for the GEMM2 items of the two one-launch modes
the share of their time spent in flag waits beside the wait their producers'
completion times imply (the latest end among the GEMM1 items that write the
Z columns the item reads, minus the item's start).  A second table gives each
mode's clock over eighths of its run.
"""
from __future__ import annotations

import argparse
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

TICK_US = 0.01  # 100 MHz device real-time counter
CAP = 128       # records per work-group


def _records(buf, G):
    """(kind, item, rank, start, main, end, ring, flag, cycles) per recorded item, sections merged."""
    import numpy as np

    a = buf.cpu().numpy().reshape(2, G, 1 + 8 * CAP)
    out = []
    for sec in (0, 1):
        for g in range(G):
            n = min(int(a[sec, g, 0]), CAP)
            for j in range(n):
                r = a[sec, g, 1 + 8 * j: 9 + 8 * j].astype(np.uint64)
                w0 = int(r[0])
                entry, rank = w0 & 0xFFFFFFFF, w0 >> 32
                # 0 GEMM1 item, 1 GEMM2 item, 2 reduction item (a slice of a split-K GEMM2 tile)
                kind = 2 if (entry & 0xC0000000) == 0xC0000000 else 1 if entry & 0x80000000 else 0
                ring, cycles = int(r[6]) & 0xFFFFFFFF, int(r[6]) >> 32
                out.append((kind, entry & 0x3FFFFFFF, rank, int(r[1]), int(r[2]), int(r[5]), ring, int(r[7]), cycles))
    return out


def _dependencies(info, F):
    """GEMM2 item -> GEMM1 tiles whose Z columns it reads (closed form of the plan).

    A plan run in row groups records the launches of a whole group, whose
    row blocks are the group's."""
    Mb = info["row_group"] // info["bm"] if info.get("row_group") else info["row_blocks"]
    S2, bn1 = info["splitk2"], info["bn1"]
    per = -(-F // S2)              # ceil(F / S2), as the plan splits K ...
    kc2 = -(-per // 64) * 64       # ... rounded up to whole 64-deep stages
    deps = {}
    for q in range(info["items2"]):
        tile, s = divmod(q, S2)
        mb = tile % Mb
        kb0, kb1 = s * kc2 // bn1, (min(F, (s + 1) * kc2) - 1) // bn1
        deps[q] = [kb * Mb + mb for kb in range(kb0, kb1 + 1)]
    return deps


def summarise(B, I, bench, key):
    import numpy as np
    import torch

    w = I.WORKLOADS[key]
    g = bench.device_random_inputs(w)
    r = bench.Runner(B, w, g, None, torch.cuda.current_stream())
    info = r.info
    G = max(info["grid_pipelined"], info["grid_gemm1"], info["grid_gemm2"])
    buf = torch.zeros(2 * G * (1 + 8 * CAP), dtype=torch.int64, device="cuda")
    # (the sentinel mode runs without row groups: a grouped plan skips it)
    modes = [(B.MODE_SEQUENTIAL, "sequential"), (B.MODE_TILE_PIPELINED, "pipelined"), (B.MODE_WORKQUEUE, "workqueue")]
    if not info["row_group"]:
        modes.append((B.MODE_SENTINEL, "sentinel"))
    for _ in range(5):
        for mode, _name in modes:
            r.run(mode)
    torch.cuda.synchronize()
    rows, clocks = [], []
    for mode, name in modes:
        buf.zero_()
        r.plan.attach_trace(buf, CAP)
        r.run(mode)
        torch.cuda.synchronize()
        r.plan.attach_trace(None, 1)
        recs = _records(buf, G)
        t0 = min(x[3] for x in recs)
        span = (max(x[5] for x in recs) - t0) * TICK_US
        clocks.append((name, span, clock_by_eighth(recs, t0)))
        for kind in (0, 1, 2):
            K = [x for x in recs if x[0] == kind]
            if not K:
                continue
            R = np.array([x[3:] for x in K], dtype=np.float64)  # start, main, end, ring, flag, cycles
            item = (R[:, 2] - R[:, 0]) * TICK_US
            main = (R[:, 1] - R[:, 0]) * TICK_US
            ring, flag = R[:, 3] * TICK_US, R[:, 4] * TICK_US
            row = {
                "mode": name, "kind": ("GEMM1", "GEMM2", "reduce")[kind], "n": len(K), "span": span,
                "item": item.mean(), "main": main.mean(), "ring": ring.mean(), "flag": flag.mean(),
                "epi": (item - main).mean(), "flag_share": flag.sum() / item.sum(),
                "kcycles": R[:, 5].mean() / 1e3, "mhz": R[:, 5].sum() / item.sum(),
            }
            if kind == 1 and name != "sequential":
                S1 = info["splitk1"]
                ready = {}
                for x in recs:
                    if x[0] == 0:
                        t = x[1] // S1
                        ready[t] = max(ready.get(t, 0), x[5])
                deps = _dependencies(info, w.F)
                exp = [max(0.0, (max(ready[t] for t in deps[x[1]]) - x[3]) * TICK_US) for x in K]
                row["implied"] = float(np.mean(exp))
            rows.append(row)
    r.check()
    r.close()
    del g
    torch.cuda.empty_cache()
    tiles = [info[k] for k in ("bm", "bn1", "splitk1", "bn2", "splitk2", "stages")]
    return w, tiles, rows, clocks


def clock_by_eighth(recs, t0):
    """Mean clock (MHz) of the items ending in each eighth of the run (cycles over real time)."""
    end = max(x[5] for x in recs)
    width = (end - t0) / 8 or 1
    out = []
    for e in range(8):
        sel = [x for x in recs if t0 + e * width <= x[5] < t0 + (e + 1) * width or (e == 7 and x[5] == end)]
        ticks = sum(x[5] - x[3] for x in sel)
        out.append(sum(x[8] for x in sel) / (ticks * TICK_US) if ticks else float("nan"))
    return out


def chain_summary(B, M: int, layers: int = 4, width: int = 8192):
    """Per layer of one traced pipelined run of the GEMM chain (GELU between
    layers, device-drawn inputs): items, mean item, mainloop and flag-wait
    times, flag share, cycles per item and clock."""
    import numpy as np
    import torch

    dims = [width] * (layers + 1)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3000 + M)
    X = torch.randn(M, width, device="cuda", generator=gen).to(torch.bfloat16)
    Ws = [(torch.randn(width, width, device="cuda", generator=gen) * width ** -0.5).to(torch.bfloat16) for _ in range(layers)]
    Y = torch.empty(M, width, dtype=torch.bfloat16, device="cuda")
    plan = B.ChainPlan(M, dims, B.ACT_GELU_TANH)
    G = plan.grid()
    buf = torch.zeros(2 * G * (1 + 8 * CAP), dtype=torch.int64, device="cuda")
    for _ in range(5):
        plan.run(X, Ws, Y, B.MODE_TILE_PIPELINED)
        plan.run(X, Ws, Y, B.MODE_SEQUENTIAL)
    torch.cuda.synchronize()
    plan.attach_trace(buf, CAP)
    plan.run(X, Ws, Y, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    plan.attach_trace(None, 1)
    assert plan.check() == B.OK
    plan.close()
    recs = _records(buf, G)
    t0 = min(x[3] for x in recs)
    span = (max(x[5] for x in recs) - t0) * TICK_US
    rows = []
    for layer in range(layers):
        K = [x for x in recs if (x[1] >> 24) == layer]
        if not K:
            continue
        R = np.array([x[3:] for x in K], dtype=np.float64)  # start, main, end, ring, flag, cycles
        item = (R[:, 2] - R[:, 0]) * TICK_US
        rows.append({"layer": layer + 1, "n": len(K), "span": span, "item": item.mean(),
                     "main": ((R[:, 1] - R[:, 0]) * TICK_US).mean(), "flag": (R[:, 4] * TICK_US).mean(),
                     "flag_share": (R[:, 4] * TICK_US).sum() / item.sum(), "kcycles": R[:, 5].mean() / 1e3,
                     "mhz": R[:, 5].sum() / item.sum(),
                     "start": ((R[:, 0] - t0) * TICK_US).min(), "end": ((R[:, 2] - t0) * TICK_US).max()})
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workloads", default="tiny,l8b_decode,l8b_prefill,l70b_gated,l70b_shard8")
    ap.add_argument("--chain-rows", default="", help="also trace the GEMM chain (4 x 8192, GELU) at these row counts")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    from paper_2607_07862_amd import binding as B
    from paper_2607_07862_amd import inputs as I
    import bench

    B.load(B.TRACE_LIB_PATH)  # the timing-trace build, chosen here and nowhere at import time
    lines = ["| workload | mode | launch µs | kind | items | item µs | mainloop µs | ring wait µs | flag wait µs | epilogue µs | flag share | producer-implied wait µs | k cycles / item | clock MHz |",
             "|---|---|---:|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    clock_lines = ["| workload | mode | launch µs | clock MHz in each eighth of the run |", "|---|---|---:|---|"]
    for key in args.workloads.split(","):
        w, tiles, rows, clocks = summarise(B, I, bench, key)
        for x in rows:
            implied = f"{x['implied']:.1f}" if "implied" in x else ""
            lines.append(f"| {key} {tiles} | {x['mode']} | {x['span']:.1f} | {x['kind']} | {x['n']} | {x['item']:.1f} | "
                         f"{x['main']:.1f} | {x['ring']:.1f} | {x['flag']:.1f} | {x['epi']:.2f} | {100 * x['flag_share']:.1f} % | {implied} | "
                         f"{x['kcycles']:.1f} | {x['mhz']:.0f} |")
        for name, span, c in clocks:
            clock_lines.append(f"| {key} | {name} | {span:.1f} | " + " ".join(f"{v:.0f}" for v in c) + " |")
        print(lines[-1] if rows else key, flush=True)
    cmd = " ".join(["python -m paper_2607_07862_amd.tracesum"] + sys.argv[1:])
    head = ["# Flag waits and where item time goes (timing-trace build, one warm run per mode)", "",
            "Command (from the repository root on the GPU host, after `python -m paper_2607_07862_amd.build --trace`):", "",
            "```", cmd, "```", "",
            "Times are means over the items of a kind; the flag share is the kind's flag-wait time over its item",
            "time (pipelined: waits on ready counters; workqueue: the wait for the popped queue slot to fill, the",
            "item starting when its work-group began to pop; sentinel: re-reads of Z pieces that still held the",
            "sentinel); the producer-implied wait is, per GEMM2 item of the",
            "one-launch modes, the latest end among the GEMM1 items writing the Z columns it reads minus its",
            "start (0 when they were done before it started).  Cycles are the item's core clock cycles",
            "(shader-clock counter); the clock is cycles over the item's real time.", ""]
    chain_lines = []
    if args.chain_rows:
        chain_lines = ["", "GEMM chain (4 layers of 8192 x 8192, GELU between), one traced pipelined run; per layer:", "",
                       "| rows | launch µs | layer | items | first start µs | last end µs | item µs | mainloop µs | flag wait µs | flag share | k cycles / item | clock MHz |",
                       "|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
        for Mc in [int(x) for x in args.chain_rows.split(",")]:
            for x in chain_summary(B, Mc):
                chain_lines.append(f"| {Mc} | {x['span']:.1f} | {x['layer']} | {x['n']} | {x['start']:.1f} | {x['end']:.1f} | "
                                   f"{x['item']:.1f} | {x['main']:.1f} | {x['flag']:.1f} | {100 * x['flag_share']:.1f} % | "
                                   f"{x['kcycles']:.1f} | {x['mhz']:.0f} |")
            print(chain_lines[-1], flush=True)
    text = "\n".join(head + lines + ["", "Clock over the run (items grouped by the eighth of the run they end in):", ""]
                     + clock_lines + chain_lines) + "\n"
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
    else:
        print(text)


if __name__ == "__main__":
    main()
