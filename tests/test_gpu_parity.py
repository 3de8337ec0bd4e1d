"""Parity of the HIP path with the fp64 oracle, through the C ABI.

* every case runs both modes; Y must be within the elementwise bound
  |Y - Y_ref| <= 2e-2 max|Y_ref| + 1e-3 and within the relative-RMS bar, and
  the two modes must agree bit for bit on Y and on the intermediate Z;
* small shapes span several tiles and a ragged row tail and are compared
  element by element against the full oracle;
* the five MLP workloads run at full size in the launch configuration the
  bench times, compared on a seeded sample of rows the oracle computes one
  by one: one row inside every row block of the plan's tiles and 24 more
  (max|Y_ref| taken over the sample, which is stricter);
* structural cases (identity and zero weights) must be bit-exact.
"""
import numpy as np
import pytest
import torch

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

from _gpu import (assert_bit_equal, assert_matches_oracle, both_modes, bits_of, device_inputs, run, sentinel_mode,
                  workqueue_mode)

pytestmark = pytest.mark.gpu

SMALL = [
    # M, H, F, act, tuning
    (1, 64, 64, 0, None),
    (7, 128, 192, 1, None),
    (33, 192, 320, 2, None),
    (100, 256, 384, 1, {"bm": 32}),
    (255, 128, 256, 0, None),
    (64, 512, 2048, 0, None),
    (130, 256, 512, 1, {"bm": 128, "splitk1": 2, "splitk2": 3}),
    (70, 320, 640, 2, {"bm": 64, "splitk1": 3, "splitk2": 2}),
    (16, 1024, 1024, 1, {"splitk1": 4, "splitk2": 4, "bn1": 64, "bn2": 64}),
    (200, 640, 1280, 1, {"bm": 128, "bn1": 128, "bn2": 128}),
    (129, 256, 384, 2, {"bm": 128, "splitk1": 2}),
    (200, 320, 640, 2, None),
    (140, 256, 384, 0, {"splitk1": 2, "splitk2": 3}),
    # 129..256 rows, SwiGLU, H a multiple of 128: the default plan's 256-row
    # tiles with the GEMM2 tile run as two halves of the GEMM1 tile's width
    (200, 1024, 1024, 2, None),
    (256, 512, 768, 2, None),
    (200, 384, 640, 2, None),
    # eight-wave work-groups: 256 x 256 tiles (two row blocks, the second ragged),
    # 256-row tiles of 128 columns, GEMM2 as two halves, the gated shapes
    (300, 512, 768, 1, {"waves": 8, "bm": 256, "bn1": 256, "bn2": 256, "stages": 2}),
    (300, 512, 768, 0, {"waves": 8, "bm": 256, "bn1": 256, "bn2": 128, "stages": 2, "splitk2": 2}),
    (257, 384, 640, 1, {"waves": 8, "bm": 256, "bn1": 128, "bn2": 128, "stages": 3, "splitk2": 2}),
    (300, 256, 512, 1, {"waves": 8, "bm": 256, "bn1": 128, "bn2": 256, "stages": 2}),
    (300, 256, 512, 2, {"waves": 8, "bm": 256, "bn1": 128, "bn2": 256, "stages": 2}),
    (200, 256, 640, 2, {"waves": 8, "bm": 256, "bn1": 64, "bn2": 128, "stages": 3, "splitk1": 2}),
    (130, 512, 1024, 1, {"waves": 8, "bm": 128, "bn1": 128, "bn2": 128, "stages": 4, "splitk1": 2, "splitk2": 2}),
    (100, 1024, 768, 0, {"waves": 8, "bm": 128, "bn1": 256, "bn2": 256, "stages": 3, "splitk1": 2}),
    (90, 256, 384, 1, {"waves": 8, "bm": 128, "bn1": 64, "bn2": 64, "stages": 4}),
    # 32-deep stages (64-byte activation rows, twice the ring depth)
    (200, 512, 640, 2, {"waves": 8, "bm": 256, "bn1": 128, "bn2": 256, "stages": 4, "bk": 32, "splitk2": 3}),
    (77, 320, 448, 0, {"bm": 128, "bn1": 64, "bn2": 64, "stages": 8, "bk": 32, "splitk2": 2}),
    (300, 256, 512, 1, {"bm": 128, "bn1": 64, "bn2": 64, "stages": 8, "bk": 32, "splitk1": 2}),
    # 128-deep stages: every GEMM2 stage reads the Z of two 64-column GEMM1
    # tiles (the consumer waits for both); split-K parts in whole stages
    (77, 256, 384, 1, {"bm": 128, "bn1": 64, "bn2": 64, "stages": 3, "bk": 128, "splitk2": 3}),
    (130, 512, 1024, 0, {"bm": 128, "bn1": 64, "bn2": 64, "stages": 3, "bk": 128, "splitk1": 2}),
    (20, 1024, 768, 1, {"bm": 32, "bn1": 64, "bn2": 128, "stages": 3, "bk": 128, "splitk1": 4, "splitk2": 2}),
    (50, 640, 1280, 1, {"bm": 32, "bn1": 64, "bn2": 64, "stages": 4, "bk": 128, "splitk2": 4}),
    (64, 384, 512, 0, {"bm": 64, "bn1": 64, "bn2": 64, "stages": 4, "bk": 128}),
    # the gated tile with non-temporal weight loads (a cache policy: same bits)
    (200, 512, 640, 2, {"waves": 8, "bm": 256, "bn1": 128, "bn2": 256, "stages": 2, "weights_nt": 1}),
]


@pytest.mark.parametrize("M,H,F,act,tuning", SMALL, ids=[f"{c[0]}x{c[1]}x{c[2]}-a{c[3]}-{c[4]}" for c in SMALL])
def test_small_shapes_against_full_oracle(lib, M, H, F, act, tuning):
    d = I.make_inputs(M, H, F, act, seed=M * 7 + H + F)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act, tuning)
    if act == 2 and 128 < M <= 256 and H % 128 == 0 and tuning is None:
        info = plan.info()
        # the GEMM2 tile runs as two halves of the GEMM1 tile's width: eight waves
        # of 128 + 128 columns where H allows, else four waves of 64 + 64
        want = (256, 256, 8) if H % 256 == 0 and F % 128 == 0 else (256, 128, 4)
        assert (info["bm"], info["bn2"], info["waves"]) == want, info
        assert info["bn2"] == 2 * info["bn1"], info
    Ys, Zs, Yp, Zp = both_modes(plan, g)
    Yq, Zq = workqueue_mode(plan, g)
    Yn = sentinel_mode(plan, g)
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp, ref, "pipelined Y")
    assert_matches_oracle(Ys, ref, "sequential Y")
    assert_bit_equal(Ys, Yp, "Y sequential vs pipelined")
    assert_bit_equal(Ys, Yn, "Y sequential vs sentinel")
    assert_bit_equal(Zs, Zp, "Z sequential vs pipelined")
    assert_bit_equal(Ys, Yq, "Y sequential vs workqueue")
    assert_bit_equal(Zs, Zq, "Z sequential vs workqueue")
    zref = O.intermediate(I.bits(d["X"]), I.bits(d["W1"]), M, H, F, act)
    assert_matches_oracle(Zp[:M], zref, "Z")
    plan.close()


def test_deep_stages_need_whole_stages_of_k(lib):
    """128-deep stages are refused where H or F is not a multiple of 128, and split-K parts round up to whole stages."""
    for M, H, F in [(64, 320, 512), (64, 512, 320)]:
        with pytest.raises(B.Mlp2Error):
            B.Plan(M, H, F, 1, {"bm": 64, "bn1": 64, "bn2": 64, "stages": 4, "bk": 128})
    plan = B.Plan(50, 640, 1280, 1, {"bm": 32, "bn1": 64, "bn2": 64, "stages": 4, "bk": 128, "splitk2": 4})
    info = plan.info()
    assert info["bk"] == 128 and info["splitk2"] == 4, info  # parts of 384, 384, 384 and 128 columns
    plan.close()


def test_weights_nt_choice(lib):
    """The non-temporal weight hint: on by itself where W1 and W2 exceed 256 MiB, off
    where they fit; forced off on request; refused where no tile is built with it."""
    w = I.WORKLOADS["l70b_gated"]
    plan = B.Plan(w.M, w.H, w.F, w.act)
    assert plan.info()["weights_nt"] == 1, plan.info()
    plan.close()
    plan = B.Plan(w.M, w.H, w.F, w.act, {"weights_nt": -1})
    assert plan.info()["weights_nt"] == 0, plan.info()
    plan.close()
    w = I.WORKLOADS["l8b_decode"]
    plan = B.Plan(w.M, w.H, w.F, w.act)
    assert plan.info()["weights_nt"] == 0, plan.info()
    plan.close()
    with pytest.raises(B.Mlp2Error):
        B.Plan(64, 256, 512, 1, {"weights_nt": 1})
    with pytest.raises(B.Mlp2Error):
        B.Plan(64, 256, 512, 1, {"weights_nt": 2})


def _workload_params():
    # the five workloads, the smallest of the paper's own shapes, one large
    # enough for the default row-band order (X + W1 above 256 MB) and one run
    # in row groups by default (Z of all rows above 256 MB)
    return [pytest.param(k, id=k) for k in I.WORKLOAD_ORDER + ["paper_m1024", "paper_m16384", "paper_m32768"]]


_cache = {}


@pytest.mark.parametrize("key", _workload_params())
def test_workloads_full_size_sampled_rows(lib, key):
    w = I.WORKLOADS[key]
    print(f"\n[parity] workload {w.name} seed {w.seed}", flush=True)
    d = I.workload_inputs(w)
    g = device_inputs(d)
    plan = B.Plan(w.M, w.H, w.F, w.act)
    Ys, Zs, Yp, Zp = both_modes(plan, g)
    assert_bit_equal(Ys, Yp, "Y sequential vs pipelined")
    assert_bit_equal(Zs, Zp, "Z sequential vs pipelined")
    Yq, Zq = workqueue_mode(plan, g)
    assert_bit_equal(Ys, Yq, "Y sequential vs workqueue")
    assert_bit_equal(Zs, Zq, "Z sequential vs workqueue")
    if not plan.info()["row_group"]:  # the sentinel mode runs without row groups
        assert_bit_equal(Ys, sentinel_mode(plan, g), "Y sequential vs sentinel")
    # one row in every row block of the plan's tiles (a grouped plan's blocks
    # tile each group, and groups are whole blocks) beside 24 seeded rows
    rows = I.sample_rows_per_block(w.M, plan.info()["bm"], 24, w.seed)
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), w.M, w.H, w.F, w.act, rows=rows)
    r = assert_matches_oracle(Yp[torch.as_tensor(rows, device="cuda")], ref, f"{w.name} sampled rows")
    print(f"[parity] {w.name}: max_abs_err={r['max_abs_err']:.4g} bound={r['bound']:.4g} rel_rms={r['rel_rms']:.3g}")
    zref = O.intermediate(I.bits(d["X"]), I.bits(d["W1"]), w.M, w.H, w.F, w.act, rows=rows)
    assert_matches_oracle(Zp[torch.as_tensor(rows, device="cuda")], zref, f"{w.name} Z sampled rows")
    plan.close()


@pytest.mark.parametrize("act", [0, 1])
@pytest.mark.parametrize("M", [37, 128])
def test_identity_weights(lib, M, act):
    """W1 = W2 = I: Y = X bit for bit (identity act); Y = bf16(gelu(X)) within the bound (GELU)."""
    H = 256
    d = I.make_inputs(M, H, H, act, seed=5)
    eye = torch.eye(H, dtype=torch.bfloat16)
    g = device_inputs({"X": d["X"], "W1": eye, "W2": eye.clone()})
    plan = B.Plan(M, H, H, act, {"splitk1": 2, "splitk2": 2})
    Ys, Zs, Yp, Zp = both_modes(plan, g)
    assert_bit_equal(Ys, Yp, "Y modes")
    if act == 0:
        assert_bit_equal(Yp, g["X"], "Y vs X")
    else:
        ref = O.gelu_tanh(O.bf16_bits_to_f64(I.bits(d["X"])))
        assert_matches_oracle(Yp, ref, "gelu(X)")
    plan.close()


@pytest.mark.parametrize("act", [0, 1, 2])
def test_zero_weights_give_exact_zero(lib, act):
    M, H, F = 50, 128, 256
    d = I.make_inputs(M, H, F, act, seed=6)
    n1 = 2 if act == 2 else 1
    g = device_inputs({"X": d["X"], "W1": torch.zeros(n1, H, F, dtype=torch.bfloat16).reshape(d["W1"].shape),
                       "W2": torch.zeros(F, H, dtype=torch.bfloat16)})
    plan = B.Plan(M, H, F, act)
    Ys, _, Yp, _ = both_modes(plan, g)
    assert np.all(bits_of(Yp) == 0) and np.all(bits_of(Ys) == 0)
    plan.close()


def test_runs_on_a_side_stream(lib):
    M, H, F, act = 96, 256, 512, 1
    d = I.make_inputs(M, H, F, act, seed=8)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        Yp = run(plan, g, B.MODE_TILE_PIPELINED, stream=s)
        Ys = run(plan, g, B.MODE_SEQUENTIAL, stream=s)
    s.synchronize()
    assert_bit_equal(Ys, Yp, "Y modes on a side stream")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp, ref, "side stream")
    plan.close()
