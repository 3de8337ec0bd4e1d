"""Row groups on the GPU: a plan run as back-to-back launches over groups of rows.

* every mode of a grouped plan gives the same bits (Y and the shared Z),
  within the oracle's bound, with and without a shorter last group, also
  when the group plans take another tile regime than one launch would;
* the automatic policy groups only once Z of all rows exceeds the 256 MB
  last-level cache (8192 x 8192 weights: 16384-row groups at 32768 rows,
  one launch at 16384 rows);
* a dropped producer signal in the whole groups' plan times out, mlp2_check
  reports it and the grouped plan recovers;
* a grouped run captured into a graph replays with the eager bits;
* at full size (20000 rows of 8192 x 8192) the automatic groups, a shorter
  last one included, match the oracle on rows around the group boundary.
"""
import numpy as np
import pytest
import torch

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

from _gpu import assert_bit_equal, assert_matches_oracle, both_modes, device_inputs, run, workqueue_mode

pytestmark = pytest.mark.gpu

CASES = [
    # M, rows per group, act: 512 + 488 rows; four groups of 256 rows (256-row tiles); 1024 + 1024 rows
    (1000, 512, 1),
    (1024, 256, 2),
    (2048, 1024, 0),
]


@pytest.mark.parametrize("M,rows,act", CASES, ids=[f"{c[0]}rows-groups{c[1]}-a{c[2]}" for c in CASES])
def test_grouped_modes_agree_and_match_the_oracle(lib, M, rows, act):
    H, F = 256, 512
    d = I.make_inputs(M, H, F, act, seed=80 + M)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"row_group": rows})
    info = plan.info()
    assert info["row_group"] == rows and info["M"] == M
    Ys, Zs, Yp, Zp = both_modes(plan, g)
    Yq, Zq = workqueue_mode(plan, g)
    assert_bit_equal(Ys, Yp, "Y sequential vs pipelined")
    assert_bit_equal(Zs, Zp, "Z sequential vs pipelined")
    assert_bit_equal(Ys, Yq, "Y sequential vs workqueue")
    assert_bit_equal(Zs, Zq, "Z sequential vs workqueue")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp, ref, "grouped Y")
    zref = O.intermediate(I.bits(d["X"]), I.bits(d["W1"]), M, H, F, act)
    assert_matches_oracle(Zp[:M], zref, "grouped Z")
    plan.close()


def test_one_launch_when_forced_or_small(lib):
    plan = B.Plan(1000, 256, 512, 1, {"row_group": -1})
    assert plan.info()["row_group"] == 0
    plan.close()
    plan = B.Plan(1000, 256, 512, 1, {"row_group": 1024})  # not fewer rows than the batch: one launch
    assert plan.info()["row_group"] == 0
    plan.close()
    with pytest.raises(B.Mlp2Error):
        B.Plan(1000, 256, 512, 1, {"row_group": 300})  # not a multiple of 256


def test_automatic_groups_follow_the_last_level_cache(lib):
    big = B.Plan(32768, 8192, 8192, 0)
    assert big.info()["row_group"] == 16384  # Z of 16384 rows x 8192 bf16 = 256 MB
    big.close()
    one = B.Plan(16384, 8192, 8192, 0)
    assert one.info()["row_group"] == 0
    one.close()


def test_grouped_option_refused_by_one_sub_plan_changes_neither(lib):
    """512-row groups take 128 x 128 tiles (two work-groups per CU), the 200-row
    rest 256-row tiles (one per CU): a grid only the groups accept is refused
    and leaves both sub-plans as they were; one both accept applies to both."""
    M, H, F, act = 712, 256, 512, 1
    d = I.make_inputs(M, H, F, act, seed=91)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"row_group": 512})
    info = plan.info()
    cus = info["num_cus"]
    assert info["row_group"] == 512 and info["occupancy"] >= 2, info
    before = info["grid_pipelined"]
    with pytest.raises(B.Mlp2Error):
        plan.set_option(B.OPT_GRID, cus + 8)  # within the groups' limit, beyond the rest's
    assert plan.info()["grid_pipelined"] == before
    Ys, _, Yp, _ = both_modes(plan, g)
    assert_bit_equal(Ys, Yp, "after the refused option")
    plan.set_option(B.OPT_GRID, cus // 2)
    assert plan.info()["grid_pipelined"] == cus // 2
    Ys2, _, Yp2, _ = both_modes(plan, g)
    assert_bit_equal(Ys, Yp2, "with a smaller grid in every sub-plan")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp2, ref, "grouped, smaller grid")
    plan.close()


def test_grouped_dropped_signal_times_out_and_recovers(lib):
    M, H, F, act = 600, 128, 256, 1
    d = I.make_inputs(M, H, F, act, seed=90)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"row_group": 256})
    plan.set_option(B.OPT_SPIN_LIMIT, 2000)
    plan.set_option(B.OPT_DROP_SIGNAL, 0)
    run(plan, g, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.ERR_TIMEOUT
    plan.set_option(B.OPT_DROP_SIGNAL, -1)
    plan.set_option(B.OPT_SPIN_LIMIT, 1 << 20)
    Yp = run(plan, g, B.MODE_TILE_PIPELINED)
    Ys = run(plan, g, B.MODE_SEQUENTIAL)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yp, "after recovery")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp, ref, "after recovery")
    plan.close()


@pytest.mark.parametrize("mode", [B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED, B.MODE_WORKQUEUE])
def test_grouped_graph_replays_match_eager_runs(lib, mode):
    """Every group's launches record into the graph; replays give the eager
    bits, also with eager runs of the other modes between them."""
    M, H, F, act = 700, 256, 512, 1
    d = I.make_inputs(M, H, F, act, seed=91)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"row_group": 256})
    ref = run(plan, g, B.MODE_SEQUENTIAL).clone()
    Y = torch.empty(M, H, dtype=torch.bfloat16, device="cuda")
    side = torch.cuda.Stream()  # default priority
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        plan.run(g["X"], g["W1"], g["W2"], Y, mode, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        plan.run(g["X"], g["W1"], g["W2"], Y, mode, stream=torch.cuda.current_stream())
    outs = []
    for i in range(6):
        Y.zero_()
        graph.replay()
        torch.cuda.synchronize()
        outs.append(Y.clone())
        run(plan, g, (B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED, B.MODE_WORKQUEUE)[i % 3])
        torch.cuda.synchronize()
    assert plan.check() == B.OK
    for n, y in enumerate(outs):
        assert_bit_equal(ref, y, f"mode {mode} replay {n}")
    del graph
    plan.close()


def test_full_size_groups_with_a_shorter_last_group(lib):
    """20000 rows of the paper's 8192 x 8192 shape: one automatic group of
    16384 rows and a last group of 3616, every mode bit-exact; the sampled
    rows straddle the group boundary and include the last row."""
    M, H, F, act = 20000, 8192, 8192, 0
    d = I.make_inputs(M, H, F, act, seed=96)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act)
    assert plan.info()["row_group"] == 16384
    Ys, Zs, Yp, Zp = both_modes(plan, g)
    assert_bit_equal(Ys, Yp, "Y sequential vs pipelined")
    assert_bit_equal(Zs, Zp, "Z sequential vs pipelined")
    Yq, _ = workqueue_mode(plan, g)
    assert_bit_equal(Ys, Yq, "Y sequential vs workqueue")
    rows = np.unique(np.concatenate([I.sample_rows(M, 12, 96), [16382, 16383, 16384, 16385, 19999]]))
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act, rows=rows)
    assert_matches_oracle(Yp[torch.as_tensor(rows, device="cuda")], ref, "rows around the group boundary")
    zref = O.intermediate(I.bits(d["X"]), I.bits(d["W1"]), M, H, F, act, rows=rows)
    assert_matches_oracle(Zp[torch.as_tensor(rows, device="cuda")], zref, "Z rows around the group boundary")
    plan.close()
