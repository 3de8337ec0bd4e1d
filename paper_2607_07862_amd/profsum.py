"""Summaries of rocprofv3 output for the committed profiles.

    python -m paper_2607_07862_amd.profsum stats DIR OUT.md --cmd "<command>"
        Kernel durations from ``--kernel-trace --stats`` CSV output in DIR.

    python -m paper_2607_07862_amd.profsum traffic FETCH_DIR WRITE_DIR WORKLOAD OUT_STEM \\
            --copy-mib N --cmd-fetch "<command>" --cmd-write "<command>"
        HBM traffic per pipelined launch from two ``--pmc`` runs (FETCH_SIZE,
        then WRITE_SIZE, KiB per dispatch), each scaled by what the same
        counter reads for the plain copy of N MiB that bench.py's
        ``--copy-calibration N`` performs first.  Writes OUT_STEM.json (read
        by bench.py, tagged with the hash of the kernel sources) and
        OUT_STEM.md.

    python -m paper_2607_07862_amd.profsum counters OUT.md DIR [DIR ...] --cmd "<command>" [--cmd ...]
        Per-kernel means of every counter of one or more ``--pmc`` runs
        (and the L2 hit rate when TCC_HIT and TCC_MISS were collected).

Reads CSV files only; runs nothing.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import re
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def short_name(n: str) -> str:
    """k_mlp2<Tile<BM, BN, WM, WN, NS[, BK[, NT]]>, NB, Tile<...>, HV, PHASE> -> phase and tile shape."""
    m = re.search(r"k_mlp2<mlp2::Tile<([^>]*)>, (\d), mlp2::Tile<([^>]*)>, (\d), (\d)>", n)
    if m:
        t1 = [x.strip() for x in m.group(1).split(",")]
        t2 = [x.strip() for x in m.group(3).split(",")]
        phase = ["gemm1", "gemm2", "pipelined", "workqueue", "sentinel"][int(m.group(5))]
        bm, bn1, wm, wn, ns = (int(x) for x in t1[:5])
        bn2 = int(t2[1]) * int(m.group(4))
        extra = ""
        if len(t1) > 5 and t1[5] != "64":
            extra += f", bk {t1[5]}"
        if len(t1) > 6 and t1[6] in ("true", "1"):
            extra += ", weights nt"
        return (f"k_mlp2 {phase} (bm {bm}, bn1 {bn1}, bn2 {bn2}, nb {m.group(2)}, stages {ns}, "
                f"waves {wm * wn}{extra})")
    return n if len(n) < 90 else n[:87] + "..."


def _one(pattern: str) -> str:
    files = sorted(glob.glob(pattern, recursive=True))
    if not files:
        sys.exit(f"no file matches {pattern}")
    return files[0]


def stats(args):
    f = _one(os.path.join(args.dir, "**", "*kernel_stats.csv"))
    rows = list(csv.DictReader(open(f)))
    lines = [
        f"# {args.title}",
        "",
        "Command (from the repository root on the GPU host):",
        "",
        "```",
        args.cmd,
        "```",
        "",
        "| kernel | calls | average µs | min µs | max µs | share of GPU time |",
        "|---|---:|---:|---:|---:|---:|",
    ]
    for r in rows:
        lines.append(
            f"| {short_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
            f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} % |"
        )
    open(args.out, "w").write("\n".join(lines) + "\n")
    print(args.out)


def _counter(dirname: str, counter: str):
    """{kernel name: [value per dispatch]} for one counter."""
    f = _one(os.path.join(dirname, "**", "*counter_collection.csv"))
    per = defaultdict(lambda: defaultdict(float))
    for r in csv.DictReader(open(f)):
        if r["Counter_Name"] != counter:
            continue
        per[r["Kernel_Name"]][r["Dispatch_Id"]] += float(r["Counter_Value"])
    return {k: list(v.values()) for k, v in per.items()}


def _copy_kernel(per: dict) -> str:
    names = [k for k in per if re.search(r"copy", k, re.I) and "k_mlp2" not in k]
    if not names:
        sys.exit("no copy kernel in the counter output (run bench.py with --copy-calibration)")
    return max(names, key=lambda k: max(per[k]))


def traffic(args):
    sys.path.insert(0, ROOT)
    from bench import kernel_source_hash
    from paper_2607_07862_amd import inputs as I

    w = I.WORKLOADS[args.workload]
    copy_bytes = args.copy_mib << 20
    out = {"workload": w.name, "kernel_source_hash": kernel_source_hash(), "copy_calibration_bytes": copy_bytes}
    lines = [f"# HBM traffic of the pipelined launch, {w.name}", ""]
    for counter, d, cmd in (("FETCH_SIZE", args.fetch_dir, args.cmd_fetch), ("WRITE_SIZE", args.write_dir, args.cmd_write)):
        per = _counter(d, counter)
        ck = _copy_kernel(per)
        copy_kib = max(per[ck])  # the largest dispatch of the copy kernel is the calibration copy
        factor = copy_bytes / (copy_kib * 1024.0)
        pk = [k for k in per if "k_mlp2" in k and re.search(r", 2>\(", k)]
        if len(pk) != 1:
            sys.exit(f"expected one pipelined kernel, found {pk}")
        vals = per[pk[0]]
        kib = sum(vals) / len(vals)
        out[counter.lower()] = {
            "kib_per_dispatch_raw": round(kib, 1),
            "dispatches": len(vals),
            "copy_kernel": short_name(ck),
            "copy_kib_raw": round(copy_kib, 1),
            "scale": round(factor, 4),
            "bytes_per_launch": int(kib * 1024 * factor),
        }
        lines += [
            f"## {counter}",
            "",
            "```",
            cmd,
            "```",
            "",
            f"- pipelined kernel: {kib:.1f} KiB per dispatch (mean of {len(vals)} dispatches)",
            f"- calibration: {short_name(ck)} copying {args.copy_mib} MiB "
            f"{'reads' if counter == 'FETCH_SIZE' else 'writes'} {copy_kib:.1f} KiB "
            f"-> scale {factor:.4f}",
            f"- scaled: {kib * 1024 * factor / 1e6:.1f} MB per launch",
            "",
        ]
    total = out["fetch_size"]["bytes_per_launch"] + out["write_size"]["bytes_per_launch"]
    out["hbm_bytes_per_launch"] = total
    out["alg_bytes"] = w.alg_bytes()
    out["ratio_to_alg"] = round(total / w.alg_bytes(), 3)
    lines += [
        f"HBM bytes per launch (fetch + write, scaled): {total / 1e6:.1f} MB; algorithmic bytes "
        f"(X + weights + Y): {w.alg_bytes() / 1e6:.1f} MB; ratio {out['ratio_to_alg']}.",
        "",
        f"Kernel sources hash: {out['kernel_source_hash']} (bench.py reports these bytes only while it matches).",
    ]
    json.dump(out, open(args.out_stem + ".json", "w"), indent=1)
    open(args.out_stem + ".md", "w").write("\n".join(lines) + "\n")
    print(args.out_stem + ".json")


def counters(args):
    """Per-kernel means (over dispatches) of every counter of one or more --pmc runs."""
    per = defaultdict(lambda: defaultdict(list))  # kernel -> counter -> values per dispatch
    for d in args.dirs:
        f = _one(os.path.join(d, "**", "*counter_collection.csv"))
        acc = defaultdict(lambda: defaultdict(float))
        for r in csv.DictReader(open(f)):
            if "k_mlp2" not in r["Kernel_Name"]:
                continue
            acc[(r["Kernel_Name"], r["Dispatch_Id"])][r["Counter_Name"]] += float(r["Counter_Value"])
        for (k, _), cs in acc.items():
            for c, v in cs.items():
                per[k][c].append(v)
    lines = [f"# {args.title}", "", "Commands (from the repository root on the GPU host), one counter pass each:", ""]
    for c in args.cmd:
        lines += ["```", c, "```", ""]
    names = sorted({c for k in per for c in per[k]})
    lines += ["| kernel | " + " | ".join(names) + " |", "|---|" + "---:|" * len(names)]
    for k in sorted(per, key=short_name):
        vals = [sum(per[k][c]) / len(per[k][c]) if per[k][c] else float("nan") for c in names]
        lines.append(f"| {short_name(k)} | " + " | ".join(f"{v:,.0f}" for v in vals) + " |")
    hit, miss = "TCC_HIT_sum", "TCC_MISS_sum"
    if hit in names and miss in names:
        lines += ["", "L2 hit rate per kernel (TCC_HIT / (TCC_HIT + TCC_MISS)):", ""]
        for k in sorted(per, key=short_name):
            if per[k][hit] and per[k][miss]:
                h, m = sum(per[k][hit]) / len(per[k][hit]), sum(per[k][miss]) / len(per[k][miss])
                lines.append(f"- {short_name(k)}: {100 * h / (h + m):.1f} %")
    lines += derived_lines(per)
    open(args.out, "w").write("\n".join(lines) + "\n")
    print(args.out)


# MI355X: 8 XCDs of 32 CUs, 4 SIMDs per CU.  GRBM_GUI_ACTIVE is collected per
# XCD and summed, so one XCD's active cycles are an eighth of it.
XCDS, CUS, SIMDS = 8, 256, 1024


def derived_lines(per) -> list:
    """Utilisations over the kernel's active cycles (per-dispatch means).

    * MFMA busy: SQ_VALU_MFMA_BUSY_CYCLES (summed over SIMDs; a
      v_mfma_f32_16x16x32_bf16 counts the 16 cycles it holds its SIMD) over
      the cycles of all 1024 SIMDs;
    * texture-data busy: TD_TD_BUSY (summed over CUs) over the cycles of all
      256 CUs;
    * wave wait share: SQ_WAIT_INST_ANY over SQ_WAVE_CYCLES (both summed over
      waves in the same units): the share of the waves' lifetimes spent
      waiting before an instruction could issue (s_waitcnt, barriers,
      dependencies).
    """
    def mean(k, c):
        v = per[k].get(c) or []
        return sum(v) / len(v) if v else None

    out = []
    for k in sorted(per, key=short_name):
        g = mean(k, "GRBM_GUI_ACTIVE")
        if not g:
            continue
        cyc = g / XCDS
        parts = []
        b = mean(k, "SQ_VALU_MFMA_BUSY_CYCLES")
        if b is not None:
            parts.append(f"MFMA busy {100 * b / (cyc * SIMDS):.1f} %")
        t = mean(k, "TD_TD_BUSY")
        if t is not None:
            parts.append(f"texture-data busy {100 * t / (cyc * CUS):.1f} %")
        wi, wc = mean(k, "SQ_WAIT_INST_ANY"), mean(k, "SQ_WAVE_CYCLES")
        if wi is not None and wc:
            parts.append(f"wave wait share {100 * wi / wc:.1f} %")
        if parts:
            out.append(f"- {short_name(k)}: " + ", ".join(parts) + f" (over {cyc:,.0f} active cycles per XCD)")
    if out:
        out = ["", "Utilisation over the kernel's active cycles (GRBM_GUI_ACTIVE / 8 per XCD; MFMA busy over "
               "1024 SIMDs, texture-data busy over 256 CUs; wave wait share: SQ_WAIT_INST_ANY over SQ_WAVE_CYCLES):",
               ""] + out
    return out


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd_name", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("out")
    s.add_argument("--cmd", required=True)
    s.add_argument("--title", default="rocprofv3 kernel statistics")
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("workload")
    t.add_argument("out_stem")
    t.add_argument("--copy-mib", type=int, required=True)
    t.add_argument("--cmd-fetch", required=True)
    t.add_argument("--cmd-write", required=True)
    c = sub.add_parser("counters")
    c.add_argument("out")
    c.add_argument("dirs", nargs="+")
    c.add_argument("--cmd", action="append", required=True)
    c.add_argument("--title", default="rocprofv3 counters")
    a = ap.parse_args()
    {"stats": stats, "traffic": traffic, "counters": counters}[a.cmd_name](a)


if __name__ == "__main__":
    main()
