"""The allocation-free entry point (``mlp2_run_noalloc``) on the GPU.

It must give the bits of ``mlp2_plan`` + ``mlp2_run`` on the same inputs (the
same tiles and the same accumulation order; only the rank tables differ),
within the oracle's bound, on consecutive calls that share the device's
static workspace, the second one smaller than the first, in every mode; and
refuse a problem whose workspace exceeds the static array.
"""
import pytest
import torch

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

from _gpu import assert_bit_equal, assert_matches_oracle, device_inputs, run

pytestmark = pytest.mark.gpu


def _with_plan(M, H, F, act, g, mode):
    plan = B.Plan(M, H, F, act)
    Y = run(plan, g, mode)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    plan.close()
    return Y


def _noalloc(M, H, act, g, mode):
    Y = torch.empty(M, H, dtype=torch.bfloat16, device="cuda")
    Y.fill_(1.0)  # every element must be overwritten
    B.run_noalloc(g["X"], g["W1"], g["W2"], Y, act, mode)
    return Y


@pytest.mark.parametrize("mode", [B.MODE_TILE_PIPELINED, B.MODE_SEQUENTIAL, B.MODE_WORKQUEUE])
def test_two_calls_in_a_row_match_the_planned_run(lib, mode):
    big = (160, 1024, 2048, 1)     # 160 rows: 256-row tiles, split-K in both GEMMs
    small = (40, 512, 1024, 2)     # then fewer rows, narrower, SwiGLU
    outs = []
    for (M, H, F, act), seed in ((big, 11), (small, 12)):
        d = I.make_inputs(M, H, F, act, seed=seed)
        g = device_inputs(d)
        Yn = _noalloc(M, H, act, g, mode)
        torch.cuda.synchronize()
        Yp = _with_plan(M, H, F, act, g, mode)
        assert_bit_equal(Yn, Yp, f"noalloc vs planned run {M}x{H}x{F}")
        ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
        assert_matches_oracle(Yn, ref, f"noalloc {M}x{H}x{F}")
        outs.append(Yn)
    # the first call's output is untouched by the second call
    assert outs[0].shape == (big[0], big[1])


def test_decode_size_matches_the_planned_run_in_each_mode(lib):
    w = I.WORKLOADS["l8b_decode"]
    d = I.workload_inputs(w)
    g = device_inputs(d)
    ref_rows = I.sample_rows(w.M, 16, w.seed)
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), w.M, w.H, w.F, w.act, rows=ref_rows)
    for mode in (B.MODE_TILE_PIPELINED, B.MODE_SEQUENTIAL):
        Yn = _noalloc(w.M, w.H, w.act, g, mode)
        Yn2 = _noalloc(w.M, w.H, w.act, g, mode)  # and once more on the same scratch
        torch.cuda.synchronize()
        Yp = _with_plan(w.M, w.H, w.F, w.act, g, mode)
        assert_bit_equal(Yn, Yp, f"decode noalloc vs planned run, mode {mode}")
        assert_bit_equal(Yn2, Yp, f"decode noalloc second call, mode {mode}")
        assert_matches_oracle(Yn[torch.as_tensor(ref_rows, device="cuda")], ref, "decode noalloc sampled rows")


def test_refuses_a_workspace_beyond_the_static_array(lib):
    M, H, F = 2048, 4096, 14336  # Z alone is 58.7 MB, with the partials beyond 64 MiB
    X = torch.zeros(M, H, dtype=torch.bfloat16, device="cuda")
    W1 = torch.zeros(H, F, dtype=torch.bfloat16, device="cuda")
    W2 = torch.zeros(F, H, dtype=torch.bfloat16, device="cuda")
    Y = torch.zeros(M, H, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.Mlp2Error) as e:
        B.run_noalloc(X, W1, W2, Y, B.ACT_GELU_TANH, B.MODE_TILE_PIPELINED)
    assert e.value.code == B.ERR_UNSUPPORTED
    rc = lib.mlp2_run_noalloc(64, 100, 128, 1, B.DTYPE_BF16, X.data_ptr(), W1.data_ptr(), W2.data_ptr(), Y.data_ptr(),
                              torch.cuda.current_stream().cuda_stream, B.MODE_SEQUENTIAL)
    assert rc == B.ERR_UNSUPPORTED  # H not a multiple of 64
    rc = lib.mlp2_run_noalloc(64, 128, 128, 1, B.DTYPE_BF16, X.data_ptr() + 2, W1.data_ptr(), W2.data_ptr(),
                              Y.data_ptr(), torch.cuda.current_stream().cuda_stream, B.MODE_SEQUENTIAL)
    assert rc == B.ERR_ALIGNMENT
