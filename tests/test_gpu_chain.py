"""The GEMM chain on the GPU, through the C ABI.

* both modes give the same bits and match the fp64 chain oracle within the
  elementwise bound, for one to four layers, ragged row counts and widths
  that differ from layer to layer;
* runs that alternate modes and inputs never read a stale intermediate or
  counter (every layer's ready counters carry over from run to run);
* with the flag waits cut to one poll a pipelined run may give up; the plan
  reports it, recovers, and its next runs are exact;
* a run captured into a graph replays with the eager bits, in both modes;
* chains wide enough for the 256 x 256 eight-wave tile (one work-group per
  CU) match the oracle over every row, ragged row counts included;
* at the paper's shape (four 8192 x 8192 layers, 4096 rows in one launch,
  16684 rows in row groups of 8192 with a shorter last one) sampled rows
  match the oracle and the modes agree bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

from _gpu import assert_bit_equal, assert_matches_oracle

pytestmark = pytest.mark.gpu

CASES = [
    # M, dims, act
    (1, [128, 128], 1),
    (100, [128, 256, 128], 1),
    (257, [256, 128, 384, 256], 1),
    (64, [128, 128, 128, 128, 128], 0),
    (300, [512, 256, 256, 512, 128], 1),
]


def _device(d):
    return d["X"].to("cuda"), [w.to("cuda") for w in d["Ws"]]


def _run(plan, X, Ws, mode):
    Y = torch.empty(plan.M, plan.dims[-1], dtype=torch.bfloat16, device="cuda")
    plan.run(X, Ws, Y, mode)
    return Y


def _oracle(d, M, dims, act, rows=None):
    return O.chain(I.bits(d["X"]), [I.bits(w) for w in d["Ws"]], M, dims, act, rows=rows)


@pytest.mark.parametrize("M,dims,act", CASES, ids=[f"{c[0]}x{'-'.join(map(str, c[1]))}-a{c[2]}" for c in CASES])
def test_modes_agree_and_match_the_oracle(lib, M, dims, act):
    d = I.chain_inputs(M, dims, seed=M + len(dims))
    X, Ws = _device(d)
    plan = B.ChainPlan(M, dims, act)
    Ys = _run(plan, X, Ws, B.MODE_SEQUENTIAL)
    Yp = _run(plan, X, Ws, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yp, "chain Y sequential vs pipelined")
    assert_matches_oracle(Yp, _oracle(d, M, dims, act), "chain Y")
    plan.close()


WIDE_CASES = [
    # M, dims, act: 16 and 9 row blocks of 256 rows (the last ragged), 256 and 288 tiles in the narrowest layer
    (4000, [256, 4096, 4096], 1),
    (2100, [384, 8192, 8192, 8192], 1),
]


@pytest.mark.parametrize("M,dims,act", WIDE_CASES, ids=[f"{c[0]}x{'-'.join(map(str, c[1]))}-a{c[2]}" for c in WIDE_CASES])
def test_wide_tiles_match_the_oracle(lib, M, dims, act):
    print(f"\n[chain wide] {M} rows, dims {dims}", flush=True)
    d = I.chain_inputs(M, dims, seed=M + 7)
    X, Ws = _device(d)
    plan = B.ChainPlan(M, dims, act)
    # the eight-wave tile runs one work-group per CU (the four-wave tiles two)
    assert plan.grid() == torch.cuda.get_device_properties(0).multi_processor_count
    Ys = _run(plan, X, Ws, B.MODE_SEQUENTIAL)
    Yp = _run(plan, X, Ws, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yp, "chain Y sequential vs pipelined")
    assert_matches_oracle(Yp, _oracle(d, M, dims, act), "chain Y")
    plan.close()


def test_alternating_modes_and_inputs(lib):
    M, dims, act = 200, [256, 384, 128, 256], 1
    ins = [I.chain_inputs(M, dims, seed=s) for s in (40, 41)]
    dev = [_device(d) for d in ins]
    plan = B.ChainPlan(M, dims, act)
    refs = [_run(plan, *dev[i], B.MODE_SEQUENTIAL).clone() for i in (0, 1)]
    torch.cuda.synchronize()
    for n in range(6):
        i = n % 2
        mode = (B.MODE_TILE_PIPELINED, B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED)[n % 3]
        Y = _run(plan, *dev[i], mode)
        torch.cuda.synchronize()
        assert plan.check() == B.OK
        assert_bit_equal(refs[i], Y, f"run {n}")
    assert_matches_oracle(refs[1], _oracle(ins[1], M, dims, act), "second inputs")
    plan.close()


def test_one_poll_waits_give_up_and_the_plan_recovers(lib):
    M, dims, act = 512, [256, 256, 256, 256, 256], 1
    d = I.chain_inputs(M, dims, seed=42)
    X, Ws = _device(d)
    plan = B.ChainPlan(M, dims, act)
    ref = _run(plan, X, Ws, B.MODE_SEQUENTIAL).clone()
    torch.cuda.synchronize()
    plan.set_spin_limit(1)
    for _ in range(3):
        _run(plan, X, Ws, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() in (B.OK, B.ERR_TIMEOUT)  # a wait that finds its producer late gives up
    assert plan.check() == B.OK  # recovered (or nothing to recover)
    plan.set_spin_limit(1 << 20)
    Y = _run(plan, X, Ws, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(ref, Y, "after recovery")
    plan.close()


GRAPH_CASES = [
    # M, dims: 64 x 64 tiles; the eight-wave 256 x 256 tile (one work-group per CU)
    (150, [128, 256, 256, 128]),
    (4000, [256, 4096, 4096]),
]


@pytest.mark.parametrize("case", range(len(GRAPH_CASES)))
@pytest.mark.parametrize("mode", [B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED])
def test_graph_replays_match_eager_runs(lib, mode, case):
    M, dims = GRAPH_CASES[case]
    act = 1
    d = I.chain_inputs(M, dims, seed=43)
    X, Ws = _device(d)
    plan = B.ChainPlan(M, dims, act)
    if case == 1:
        assert plan.grid() == torch.cuda.get_device_properties(0).multi_processor_count
    ref = _run(plan, X, Ws, B.MODE_SEQUENTIAL).clone()
    Y = torch.empty(M, dims[-1], dtype=torch.bfloat16, device="cuda")
    side = torch.cuda.Stream()  # default priority
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        plan.run(X, Ws, Y, mode, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        plan.run(X, Ws, Y, mode, stream=torch.cuda.current_stream())
    outs = []
    for i in range(4):
        Y.zero_()
        graph.replay()
        torch.cuda.synchronize()
        outs.append(Y.clone())
        _run(plan, X, Ws, (B.MODE_SEQUENTIAL, B.MODE_TILE_PIPELINED)[i % 2])
        torch.cuda.synchronize()
    assert plan.check() == B.OK
    for n, y in enumerate(outs):
        assert_bit_equal(ref, y, f"mode {mode} replay {n}")
    del graph
    plan.close()


def test_argument_errors(lib):
    with pytest.raises(B.Mlp2Error):
        B.ChainPlan(64, [128, 100], 1)  # widths must be multiples of 128
    with pytest.raises(B.Mlp2Error):
        B.ChainPlan(64, [128, 128], 2)  # SwiGLU is not a chain activation
    with pytest.raises(B.Mlp2Error):
        B.ChainPlan(64, [128] * 10, 1)  # at most 8 layers
    plan = B.ChainPlan(64, [128, 128, 128], 1)
    d = I.chain_inputs(64, [128, 128, 128], seed=44)
    X, Ws = _device(d)
    Y = torch.empty(64, 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.Mlp2Error):
        plan.run(X, Ws, Y, B.MODE_WORKQUEUE)
    with pytest.raises(B.Mlp2Error):
        plan.run(X, Ws, X, B.MODE_SEQUENTIAL)  # Y over X
    plan.close()


@pytest.mark.parametrize("M", [4096, 16684])
def test_paper_shape_four_layers_sampled_rows(lib, M):
    """4096 rows run as one launch per mode; 16684 rows in two row groups of
    8192 and a last group of 300 (the sampled rows include both sides of the
    group boundaries and the last row)."""
    dims, act = [8192] * 5, 1
    print(f"\n[chain] {M} rows, dims {dims}", flush=True)
    d = I.chain_inputs(M, dims, seed=45)
    X, Ws = _device(d)
    plan = B.ChainPlan(M, dims, act)
    Ys = _run(plan, X, Ws, B.MODE_SEQUENTIAL)
    Yp = _run(plan, X, Ws, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yp, "chain Y sequential vs pipelined")
    rows = np.unique(np.concatenate([I.sample_rows(M, 12, 45), [min(8191, M - 1), min(8192, M - 1), min(16383, M - 1), min(16384, M - 1), M - 1]]))
    ref = _oracle(d, M, dims, act, rows=rows)
    assert_matches_oracle(Yp[torch.as_tensor(rows, device="cuda")], ref, "sampled rows")
    plan.close()
