"""The pipelining protocol on the GPU: ordering, counter lifetime, failure.

* any GEMM1 tile order and any persistent grid size give the sequential
  mode's bits (the consumer waits for exactly the producer tiles it reads;
  Sec. III-A: a consumer runs once all its producers are complete);
* runs that alternate inputs and modes never read a stale intermediate and
  never see a counter from an earlier run (the ready counters, split-K
  counters and the epoch carry over from run to run without host resets);
* a dropped producer signal (failure injection from the host) makes the
  bounded wait give up, every kernel still exits, mlp2_check reports the
  timeout and the plan recovers; so does one beyond the first 64 column
  blocks of a consumer whose first 64 are all ready (the wait reads
  readiness 64 blocks at a time);
* the workqueue mode (scoreboards and a device queue) gives the same bits;
* so do the stage splits of the pipelined launch: the rank-table lag at its
  extremes (one rank; every GEMM2 item after every GEMM1 item) and static
  producer / consumer role splits of the grid;
* a run captured into a graph replays with the eager bits, in every mode;
* the sentinel mode (no fence, no flag: consumers re-read the intermediate
  until no sentinel is left) gives the same bits, alternating with the other
  modes; a dropped tile times out and the plan recovers; the sentinel value
  is never an output of the epilogue.
"""
import pytest
import torch

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

from _gpu import assert_bit_equal, assert_matches_oracle, bits_of, device_inputs, run

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("order", [B.ORDER_AUTO, B.ORDER_ROW_FIRST, B.ORDER_REVERSED, B.ORDER_SHUFFLED,
                                   B.ORDER_COLUMN_FIRST, B.ORDER_BANDED])
@pytest.mark.parametrize("grid", [1, 2, 3, 4, 17, 0])
def test_orders_and_grids_match_sequential_bits(lib, order, grid):
    M, H, F, act = 160, 256, 768, 1
    d = I.make_inputs(M, H, F, act, seed=40 + order)
    g = device_inputs(d)
    # split-K 1 for the banded order (bands apply to unsplit GEMM1 tiles), else 2 and 3
    tun = {"bm": 32, "splitk1": 1, "splitk2": 1} if order == B.ORDER_BANDED else {"bm": 64, "splitk1": 2, "splitk2": 3}
    plan = B.Plan(M, H, F, act, tun)
    Ys = run(plan, g, B.MODE_SEQUENTIAL).clone()
    plan.set_option(B.OPT_ORDER, order)
    if grid:
        plan.set_option(B.OPT_GRID, grid)
    Yp = run(plan, g, B.MODE_TILE_PIPELINED).clone()
    Yq = run(plan, g, B.MODE_WORKQUEUE)
    Ys2 = run(plan, g, B.MODE_SEQUENTIAL)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yp, f"order {order} grid {grid}")
    assert_bit_equal(Ys, Yq, f"order {order} grid {grid} workqueue")
    assert_bit_equal(Ys, Ys2, f"order {order} grid {grid} sequential after the order change")
    plan.close()


# The stage split of the pipelined launch: the rank-table lag (shared roles)
# at its extremes, and static role splits of the grid, on a shape whose GEMM1
# spans several rounds of the grid (so consumers really wait on producers).
SPLITS = [
    {"lag": 1}, {"lag": -1}, {"lag": 100000}, {"lag": 37},
    {"p1": 8}, {"p1": 32}, {"p1": 56},
    {"p1": 32, "waves": 8, "bm": 256, "bn1": 256, "bn2": 256, "stages": 2},
    {"lag": 1, "waves": 8, "bm": 256, "bn1": 128, "bn2": 128, "stages": 3, "splitk2": 2},
]


@pytest.mark.parametrize("tuning", SPLITS, ids=[",".join(f"{k}{v}" for k, v in t.items()) for t in SPLITS])
@pytest.mark.parametrize("grid", [0, 60])
def test_stage_splits_match_sequential_bits(lib, tuning, grid):
    M, H, F, act = 600, 512, 1536, 1
    d = I.make_inputs(M, H, F, act, seed=77)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, tuning)
    info = plan.info()
    assert info["p1"] == tuning.get("p1", 0)
    if "lag" in tuning and tuning["lag"] > 0:
        assert info["lag"] == tuning["lag"]
    if tuning.get("lag") == -1:
        assert info["lag"] == info["items1"]
    if grid:
        plan.set_option(B.OPT_GRID, grid)
    Ys = run(plan, g, B.MODE_SEQUENTIAL).clone()
    Yp = run(plan, g, B.MODE_TILE_PIPELINED).clone()
    Yp2 = run(plan, g, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yp, f"{tuning} grid {grid}")
    assert_bit_equal(Ys, Yp2, f"{tuning} grid {grid}, second run")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp, ref, f"{tuning}")
    plan.close()


def test_role_split_needs_both_roles(lib):
    with pytest.raises(B.Mlp2Error):
        B.Plan(64, 128, 128, 1, {"p1": 12})  # not a multiple of 8
    plan = B.Plan(600, 512, 1536, 1, {"p1": 32})
    with pytest.raises(B.Mlp2Error):
        plan.set_option(B.OPT_GRID, 1)  # one work-group cannot hold both roles
    with pytest.raises(B.Mlp2Error):
        plan.set_option(B.OPT_GRID, 32)  # 32 work-groups: all of them in the GEMM1 role
    plan.set_option(B.OPT_GRID, 40)  # 32 + 8
    plan.close()


def test_stage_modes_compose_the_sequential_mode(lib):
    """STAGE1 then STAGE2 (same stream, or two streams ordered by an event, as a
    micro-batch pipeline schedules them) give the sequential mode's bits, also
    interleaved with runs of the other modes; grouped plans refuse them."""
    M, H, F, act = 300, 512, 1024, 1
    d = I.make_inputs(M, H, F, act, seed=31)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act)
    Ys = run(plan, g, B.MODE_SEQUENTIAL).clone()
    Y1 = torch.empty_like(Ys)
    run(plan, g, B.MODE_STAGE1, Y=Y1)
    run(plan, g, B.MODE_STAGE2, Y=Y1)
    Yp = run(plan, g, B.MODE_TILE_PIPELINED).clone()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    Y2 = torch.empty_like(Ys)
    done1 = torch.cuda.Event()
    with torch.cuda.stream(s1):
        run(plan, g, B.MODE_STAGE1, Y=Y2, stream=s1)
        done1.record(s1)
    s2.wait_event(done1)
    with torch.cuda.stream(s2):
        run(plan, g, B.MODE_STAGE2, Y=Y2, stream=s2)
    s2.synchronize()
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Y1, "stages on one stream")
    assert_bit_equal(Ys, Y2, "stages on two streams")
    assert_bit_equal(Ys, Yp, "pipelined after the stages")
    plan.close()
    grouped = B.Plan(600, 128, 256, 1, {"row_group": 256})
    gg = device_inputs(I.make_inputs(600, 128, 256, 1, seed=32))
    with pytest.raises(B.Mlp2Error) as e:
        run(grouped, gg, B.MODE_STAGE1)
    assert e.value.code == B.ERR_UNSUPPORTED
    grouped.close()


@pytest.mark.parametrize("act", [0, 1, 2])
def test_alternating_inputs_and_modes(lib, act):
    M, H, F = 96, 256, 512
    sets = [device_inputs(I.make_inputs(M, H, F, act, seed=60 + i)) for i in range(3)]
    plan = B.Plan(M, H, F, act, {"bm": 32, "splitk1": 2, "splitk2": 2})
    refs = []
    for gi in sets:
        refs.append(run(plan, gi, B.MODE_SEQUENTIAL).clone())
    torch.cuda.synchronize()
    outs = []
    seq = [0, 1, 2, 2, 0, 1, 0, 0, 2, 1] * 3
    modes = (B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED, B.MODE_WORKQUEUE, B.MODE_SENTINEL, B.MODE_SENTINEL,
             B.MODE_TILE_PIPELINED, B.MODE_SENTINEL)
    for n, i in enumerate(seq):
        mode = modes[n % len(modes)]
        outs.append((i, run(plan, sets[i], mode)))
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    for n, (i, y) in enumerate(outs):
        assert_bit_equal(y, refs[i], f"run {n} (inputs {i})")
    plan.close()


def test_repeated_pipelined_runs_are_bit_stable(lib):
    w = I.WORKLOADS["tiny"]
    g = device_inputs(I.workload_inputs(w))
    plan = B.Plan(w.M, w.H, w.F, w.act)
    first = run(plan, g, B.MODE_TILE_PIPELINED).clone()
    ys = [run(plan, g, B.MODE_TILE_PIPELINED) for _ in range(200)]
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    ref = bits_of(first)
    for n, y in enumerate(ys):
        assert (bits_of(y) == ref).all(), f"run {n}"
    plan.close()


def test_dropped_signal_times_out_and_recovers(lib):
    M, H, F, act = 64, 128, 256, 1
    d = I.make_inputs(M, H, F, act, seed=70)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act)
    plan.set_option(B.OPT_SPIN_LIMIT, 2000)
    plan.set_option(B.OPT_DROP_SIGNAL, 0)
    run(plan, g, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.ERR_TIMEOUT
    # recovered: counters reset, the next runs are correct in both modes
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


def test_sentinel_mode_dropped_tile_times_out_and_recovers(lib):
    """Sentinel mode: a GEMM1 tile whose intermediate stores are skipped leaves
    sentinels that its consumers keep re-reading until the bounded wait gives
    up; every kernel still exits, mlp2_check reports the timeout and refills
    both sentinel intermediates, and the following runs of every mode (two
    sentinel runs: both intermediates) are correct."""
    M, H, F, act = 130, 256, 512, 1
    d = I.make_inputs(M, H, F, act, seed=71)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"splitk1": 2})
    plan.set_option(B.OPT_SPIN_LIMIT, 200)
    plan.set_option(B.OPT_DROP_SIGNAL, 1)
    run(plan, g, B.MODE_SENTINEL)
    torch.cuda.synchronize()
    assert plan.check() == B.ERR_TIMEOUT
    plan.set_option(B.OPT_DROP_SIGNAL, -1)
    plan.set_option(B.OPT_SPIN_LIMIT, 1 << 20)
    Ys = run(plan, g, B.MODE_SEQUENTIAL).clone()
    Yn1 = run(plan, g, B.MODE_SENTINEL).clone()
    Yn2 = run(plan, g, B.MODE_SENTINEL).clone()
    Yp = run(plan, g, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    for y, what in ((Yn1, "sentinel run 1"), (Yn2, "sentinel run 2"), (Yp, "pipelined")):
        assert_bit_equal(Ys, y, f"after recovery: {what}")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yn2, ref, "after recovery")
    plan.close()


def test_sentinel_value_is_never_an_output(lib):
    """The epilogue turns the sentinel pattern into the canonical NaN in every
    mode: X holding NaNs whose bf16 pattern is 0xFFFF gives no 0xFFFF in Z,
    and the modes still agree bit for bit (identity weights pass X through)."""
    M, H = 64, 128
    X = torch.randn(M, H).to(torch.bfloat16)
    xb = X.view(torch.int16)
    xb[3, 5] = -1  # 0xFFFF
    xb[10, 64] = -1
    eye = torch.eye(H, dtype=torch.bfloat16)
    g = device_inputs({"X": X, "W1": eye, "W2": eye.clone()})
    plan = B.Plan(M, H, H, 0)
    outs = {}
    for mode in (B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED, B.MODE_SENTINEL):
        outs[mode] = run(plan, g, mode).clone()
        torch.cuda.synchronize()
        Z = bits_of(plan.intermediate())
        if mode != B.MODE_SENTINEL:
            assert not (Z == 0xFFFF).any()
    assert plan.check() == B.OK
    assert_bit_equal(outs[B.MODE_SEQUENTIAL], outs[B.MODE_SENTINEL], "sentinel mode with NaN inputs")
    assert_bit_equal(outs[B.MODE_SEQUENTIAL], outs[B.MODE_TILE_PIPELINED], "pipelined mode with NaN inputs")
    plan.close()


@pytest.mark.parametrize("dropped", [63, 64, 80, 99])
def test_wait_covers_blocks_past_one_full_window(lib, dropped):
    """A consumer whose first 64 column blocks are all ready still waits for later ones.

    One work-group runs every GEMM1 item before the single GEMM2 item, whose
    K range covers 100 column blocks; when it starts, every block but the
    dropped one is ready, so its first gather finds a full 64-block window.
    The missing signal must end in a time-out, never in a skipped wait.
    """
    M, H, F, act = 32, 64, 6400, 1
    d = I.make_inputs(M, H, F, act, seed=71)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"bm": 32, "bn1": 64, "splitk1": 1, "bn2": 64, "splitk2": 1})
    info = plan.info()
    assert (info["items1"], info["items2"], info["row_blocks"]) == (100, 1, 1)
    plan.set_option(B.OPT_GRID, 1)
    plan.set_option(B.OPT_SPIN_LIMIT, 2000)
    plan.set_option(B.OPT_DROP_SIGNAL, dropped)
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
    plan.close()


@pytest.mark.parametrize("s2", [1, 2])
@pytest.mark.parametrize("grid", [0, 1, 5, 24])
def test_xcd_grouped_default_order(lib, grid, s2):
    """Several row blocks: the default order deals the GEMM1 tiles to the XCDs
    in sub-blocks (ragged here: 5 row blocks), and the GEMM2 tiles too
    without split-K (with it, GEMM2 items go in item order).  The pipelined
    mode gives the sequential mode's bits, within the oracle's bound."""
    M, H, F, act = 640, 256, 1024, 1
    d = I.make_inputs(M, H, F, act, seed=90)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"bm": 128, "bn1": 128, "bn2": 128, "splitk1": 1, "splitk2": s2})
    info = plan.info()
    assert (info["row_blocks"], info["splitk1"], info["splitk2"], info["order"]) == (5, 1, s2, B.ORDER_AUTO)
    if grid:
        plan.set_option(B.OPT_GRID, grid)
    Ys = run(plan, g, B.MODE_SEQUENTIAL).clone()
    Yp = run(plan, g, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yp, f"grid {grid}")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp, ref, f"grid {grid}")
    plan.close()


WQ_CASES = [
    # M, H, F, act, tuning
    (160, 256, 768, 1, {"bm": 64, "splitk1": 2, "splitk2": 3}),
    (96, 256, 512, 0, {"bm": 32, "splitk1": 1, "splitk2": 2}),
    (256, 1024, 4096, 2, {"bm": 128, "bn1": 64, "bn2": 128, "splitk2": 2}),
    (640, 256, 1024, 1, {"bm": 128, "bn1": 128, "bn2": 128, "splitk1": 1, "splitk2": 1}),
    # K ranges of 192 across 128-column blocks: one GEMM1 tile feeds two parts of each GEMM2 tile
    (64, 256, 1152, 1, {"bm": 64, "bn1": 128, "bn2": 64, "splitk2": 6}),
]


@pytest.mark.parametrize("case", range(len(WQ_CASES)))
@pytest.mark.parametrize("grid", [1, 3, 0])
def test_workqueue_mode_matches_sequential_bits(lib, case, grid):
    """The paper's scoreboard-and-workqueue scheduling (Sec. III-A.2-3) gives
    the sequential mode's bits for any grid, split-K and activation."""
    M, H, F, act, tun = WQ_CASES[case]
    d = I.make_inputs(M, H, F, act, seed=100 + case)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, tun)
    Ys = run(plan, g, B.MODE_SEQUENTIAL).clone()
    if grid:
        plan.set_option(B.OPT_GRID, grid)
    outs = [run(plan, g, B.MODE_WORKQUEUE).clone() for _ in range(3)]
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    for n, y in enumerate(outs):
        assert_bit_equal(Ys, y, f"case {case} grid {grid} run {n}")
    if case == 4 and grid == 0:
        ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
        assert_matches_oracle(outs[0], ref, "workqueue")
    plan.close()


def test_workqueue_dropped_signal_times_out_and_recovers(lib):
    M, H, F, act = 64, 128, 256, 1
    d = I.make_inputs(M, H, F, act, seed=72)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act)
    plan.set_option(B.OPT_SPIN_LIMIT, 2000)
    plan.set_option(B.OPT_DROP_SIGNAL, 0)
    run(plan, g, B.MODE_WORKQUEUE)
    torch.cuda.synchronize()
    assert plan.check() == B.ERR_TIMEOUT
    plan.set_option(B.OPT_DROP_SIGNAL, -1)
    plan.set_option(B.OPT_SPIN_LIMIT, 1 << 20)
    Yq = run(plan, g, B.MODE_WORKQUEUE).clone()
    Ys = run(plan, g, B.MODE_SEQUENTIAL)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yq, "after recovery")
    plan.close()


@pytest.mark.parametrize("mode", [B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED, B.MODE_WORKQUEUE, B.MODE_SENTINEL])
def test_graph_replays_match_eager_runs(lib, mode):
    """mlp2_run records into a graph (kernel launches only: no memset, no
    synchronisation), and every replay gives the eager bits: the counters and
    epochs live on the device and advance once per replay, also with eager
    runs of the other modes between the replays."""
    M, H, F, act = 96, 256, 512, 1
    d = I.make_inputs(M, H, F, act, seed=95)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"bm": 32, "splitk1": 2, "splitk2": 2})
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
        run(plan, g, (B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED, B.MODE_WORKQUEUE, B.MODE_SENTINEL)[i % 4])
        torch.cuda.synchronize()
    assert plan.check() == B.OK
    for n, y in enumerate(outs):
        assert_bit_equal(ref, y, f"mode {mode} replay {n}")
    del graph
    plan.close()


def test_run_argument_errors(lib):
    M, H, F = 32, 64, 128
    g = device_inputs(I.make_inputs(M, H, F, 0, seed=1))
    plan = B.Plan(M, H, F, 0)
    Y = torch.empty(M, H, dtype=torch.bfloat16, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    X, W1, W2, y = (t.data_ptr() for t in (g["X"], g["W1"], g["W2"], Y))
    assert plan.run_raw(X, W1, W2, y, s, 6) == B.ERR_INVALID_ARG
    assert plan.run_raw(X, W1, W2, y, s, -1) == B.ERR_INVALID_ARG
    assert plan.run_raw(X + 2, W1, W2, y, s, 0) == B.ERR_ALIGNMENT
    assert plan.run_raw(X, W1, W2, X, s, 0) == B.ERR_INVALID_ARG  # Y aliases X
    assert plan.run_raw(0, W1, W2, y, s, 0) == B.ERR_INVALID_ARG
    with pytest.raises(ValueError):
        plan.run(g["X"], g["W1"], g["W2"], torch.empty(M, H + 1, dtype=torch.bfloat16, device="cuda"), 0)
    info = plan.info()
    assert info["items1"] == info["row_blocks"] * info["col_blocks1"] * info["splitk1"]
    # persistent grids: any size from one work-group up to what fits the device at once
    too_many = info["occupancy"] * info["num_cus"] + 1
    with pytest.raises(B.Mlp2Error):
        plan.set_option(B.OPT_GRID, too_many)
    with pytest.raises(B.Mlp2Error):
        plan.set_option(B.OPT_GRID, -1)
    plan.set_option(B.OPT_GRID, 1)
    plan.set_option(B.OPT_GRID, 0)
    assert info["grid_pipelined"] >= 1 and info["occupancy"] >= 1
    plan.close()


@pytest.mark.parametrize("order", [B.ORDER_REVERSED, B.ORDER_SHUFFLED, B.ORDER_COLUMN_FIRST, B.ORDER_AUTO])
def test_consecutive_slice_waits_stay_in_step(lib, order):
    """bn1 = 64 makes every 64-deep stage of GEMM2 a new column block of Z, so
    the pipeline prologue waits several times in a row; with a reversed or
    shuffled GEMM1 order those waits see short ready prefixes.  Every run must
    give the sequential mode's bits."""
    M, H, F, act = 256, 1024, 4096, 2
    d = I.make_inputs(M, H, F, act, seed=80 + order)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, {"bm": 128, "bn1": 64, "bn2": 128, "splitk2": 2})
    Ys = run(plan, g, B.MODE_SEQUENTIAL).clone()
    plan.set_option(B.OPT_ORDER, order)
    outs = [run(plan, g, B.MODE_TILE_PIPELINED) for _ in range(20)]
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    for n, y in enumerate(outs):
        assert_bit_equal(Ys, y, f"run {n}")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Ys, ref, "sequential")
    plan.close()
