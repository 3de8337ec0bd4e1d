"""The rocprofv3 summariser on synthetic CSV files (host logic only).

* demangled kernel names shorten to their phase and tile shape (the gated
  GEMM2 halves counted into bn2);
* the traffic summary scales each counter by what it reads for the copy
  kernel of known size, averages the pipelined kernel's dispatches and
  compares with the workload's algorithmic bytes, under the current kernel
  sources' hash;
* the statistics table carries every kernel row with times in microseconds.
"""
import argparse
import csv
import json
import os

import pytest

from paper_2607_07862_amd import inputs as I
from paper_2607_07862_amd import profsum as P

PIPE = "void mlp2::k_mlp2<mlp2::Tile<128, 64, 2, 2, 4>, 1, mlp2::Tile<128, 64, 2, 2, 4>, 1, 2>(mlp2::Args)"
GATED2 = "void mlp2::k_mlp2<mlp2::Tile<256, 64, 4, 1, 3>, 2, mlp2::Tile<256, 64, 4, 1, 3>, 2, 1>(mlp2::Args)"
COPY = "__amd_rocclr_copyBuffer"


def test_short_names():
    assert P.short_name(PIPE) == "k_mlp2 pipelined (bm 128, bn1 64, bn2 64, nb 1, stages 4, waves 4)"
    assert P.short_name(GATED2) == "k_mlp2 gemm2 (bm 256, bn1 64, bn2 128, nb 2, stages 3, waves 4)"
    wide = "void mlp2::k_mlp2<mlp2::Tile<256, 256, 2, 4, 2>, 1, mlp2::Tile<256, 256, 2, 4, 2>, 1, 2>(mlp2::Args)"
    assert P.short_name(wide) == "k_mlp2 pipelined (bm 256, bn1 256, bn2 256, nb 1, stages 2, waves 8)"
    # the stage depth as a sixth tile parameter (named only when it is not 64), the sentinel phase
    deep = "void mlp2::k_mlp2<mlp2::Tile<256, 128, 4, 2, 2, 64>, 2, mlp2::Tile<256, 128, 4, 2, 2, 64>, 2, 4>(mlp2::Args)"
    assert P.short_name(deep) == "k_mlp2 sentinel (bm 256, bn1 128, bn2 256, nb 2, stages 2, waves 8)"
    bk32 = "void mlp2::k_mlp2<mlp2::Tile<128, 64, 2, 2, 8, 32>, 1, mlp2::Tile<128, 64, 2, 2, 8, 32>, 1, 3>(mlp2::Args)"
    assert P.short_name(bk32) == "k_mlp2 workqueue (bm 128, bn1 64, bn2 64, nb 1, stages 8, waves 4, bk 32)"
    # the non-temporal weight hint as a seventh tile parameter
    nt = "void mlp2::k_mlp2<mlp2::Tile<256, 128, 4, 2, 2, 64, true>, 2, mlp2::Tile<256, 128, 4, 2, 2, 64, true>, 2, 2>(mlp2::Args)"
    assert P.short_name(nt) == "k_mlp2 pipelined (bm 256, bn1 128, bn2 256, nb 2, stages 2, waves 8, weights nt)"
    off = "void mlp2::k_mlp2<mlp2::Tile<128, 64, 2, 2, 4, 64, false>, 1, mlp2::Tile<128, 64, 2, 2, 4, 64, false>, 1, 0>(mlp2::Args)"
    assert P.short_name(off) == "k_mlp2 gemm1 (bm 128, bn1 64, bn2 64, nb 1, stages 4, waves 4)"
    assert P.short_name("x" * 200).endswith("...")


def _counters(path, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], r)))


def test_traffic_scales_by_the_copy_calibration(tmp_path):
    fetch, write = str(tmp_path / "fetch"), str(tmp_path / "write")
    # the 256 MiB copy reads 131072 KiB (a factor of 2 to the bytes copied); two pipelined dispatches
    _counters(fetch, [(1, COPY, "FETCH_SIZE", 131072), (2, PIPE, "FETCH_SIZE", 100000), (3, PIPE, "FETCH_SIZE", 110000),
                      (3, PIPE, "OTHER", 5)])
    _counters(write, [(1, COPY, "WRITE_SIZE", 262144), (2, PIPE, "WRITE_SIZE", 10000), (3, PIPE, "WRITE_SIZE", 10000)])
    stem = str(tmp_path / "traffic")
    P.traffic(argparse.Namespace(fetch_dir=fetch, write_dir=write, workload="l8b_decode", out_stem=stem, copy_mib=256,
                                 cmd_fetch="fetch cmd", cmd_write="write cmd"))
    out = json.load(open(stem + ".json"))
    assert out["fetch_size"]["scale"] == pytest.approx(2.0)
    assert out["fetch_size"]["bytes_per_launch"] == int(105000 * 1024 * 2.0)
    assert out["write_size"]["scale"] == pytest.approx(1.0)
    assert out["hbm_bytes_per_launch"] == int(105000 * 1024 * 2.0) + int(10000 * 1024)
    assert out["alg_bytes"] == I.WORKLOADS["l8b_decode"].alg_bytes()
    import bench
    assert out["kernel_source_hash"] == bench.kernel_source_hash()
    text = open(stem + ".md").read()
    assert "fetch cmd" in text and "write cmd" in text and "mean of 2 dispatches" in text


def test_stats_table(tmp_path):
    d = tmp_path / "kt" / "host"
    d.mkdir(parents=True)
    with open(d / "run_kernel_stats.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "AverageNs", "MinNs", "MaxNs", "Percentage"])
        w.writeheader()
        w.writerow({"Name": PIPE, "Calls": 10, "AverageNs": 75000, "MinNs": 70000, "MaxNs": 90000, "Percentage": 61.5})
    out = str(tmp_path / "stats.md")
    P.stats(argparse.Namespace(dir=str(tmp_path / "kt"), out=out, cmd="the cmd", title="t"))
    text = open(out).read()
    assert "| k_mlp2 pipelined (bm 128, bn1 64, bn2 64, nb 1, stages 4, waves 4) | 10 | 75.00 | 70.00 | 90.00 | 61.5 % |" in text
    assert "the cmd" in text


def test_counter_utilisations(tmp_path):
    # two dispatches of 1000 cycles per XCD; MFMA busy half of every SIMD's cycles,
    # the texture-data units a quarter of every CU's, the waves waiting 30 % of their
    # cycles in one dispatch and 20 % in the other; two passes merged per kernel
    a, b = str(tmp_path / "mfma"), str(tmp_path / "path")
    _counters(a, [(1, PIPE, "GRBM_GUI_ACTIVE", 8000), (1, PIPE, "SQ_VALU_MFMA_BUSY_CYCLES", 1024 * 500),
                  (1, PIPE, "SQ_WAIT_INST_ANY", 360), (1, PIPE, "SQ_WAVE_CYCLES", 1200),
                  (2, PIPE, "GRBM_GUI_ACTIVE", 8000), (2, PIPE, "SQ_VALU_MFMA_BUSY_CYCLES", 1024 * 500),
                  (2, PIPE, "SQ_WAIT_INST_ANY", 240), (2, PIPE, "SQ_WAVE_CYCLES", 1200),
                  (3, COPY, "GRBM_GUI_ACTIVE", 10)])
    _counters(b, [(5, PIPE, "GRBM_GUI_ACTIVE", 8000), (5, PIPE, "TD_TD_BUSY", 256 * 250)])
    out = str(tmp_path / "c.md")
    P.counters(argparse.Namespace(dirs=[a, b], out=out, cmd=["pass 1", "pass 2"], title="t"))
    text = open(out).read()
    assert ("- k_mlp2 pipelined (bm 128, bn1 64, bn2 64, nb 1, stages 4, waves 4): MFMA busy 50.0 %, "
            "texture-data busy 25.0 %, wave wait share 25.0 % (over 1,000 active cycles per XCD)") in text
    assert "pass 1" in text and "pass 2" in text and COPY not in text
