"""The size limits on the GPU.

* the largest row count (2^20 rows) and the largest widths (F = 2^18 and
  H = 2^18 at 32 rows) that the plan accepts run in every mode, bit-exact
  across modes and within the oracle's bound (sampled rows at 2^20 rows);
* operands of 4 GB or more per launch (X, Z, a weight matrix), which the
  loads' 32-bit byte offsets cannot address, are refused at plan time, and
  so are sizes outside the documented ranges; a batch whose X exceeds 4 GB
  but runs in row groups is accepted (each group's X is a slice);
* the chain refuses the same.
"""
import pytest
import torch

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

from _gpu import assert_bit_equal, assert_matches_oracle, both_modes, device_inputs, workqueue_mode

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,H,F,act,sampled", [
    (1 << 20, 64, 64, 1, True),
    (32, 64, 1 << 18, 1, False),
    (32, 1 << 18, 64, 0, False),
], ids=["rows-2^20", "F-2^18", "H-2^18"])
def test_largest_accepted_sizes(lib, M, H, F, act, sampled):
    print(f"\n[limits] M={M} H={H} F={F}", flush=True)
    d = I.make_inputs(M, H, F, act, seed=97)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act)
    Ys, Zs, Yp, Zp = both_modes(plan, g)
    assert_bit_equal(Ys, Yp, "Y sequential vs pipelined")
    Yq, _ = workqueue_mode(plan, g)
    assert_bit_equal(Ys, Yq, "Y sequential vs workqueue")
    rows = I.sample_rows(M, 24, 97) if sampled else None
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act, rows=rows)
    got = Yp[torch.as_tensor(rows, device="cuda")] if sampled else Yp
    assert_matches_oracle(got, ref, "largest sizes")
    plan.close()


@pytest.mark.parametrize("M,H,F,act", [
    (1 << 20, 4096, 64, 1),      # X of 8 GB, one launch (Z is small, so no row groups)
    (64, 1 << 16, 1 << 15, 1),   # W1 of 4 GB
    (64, 1 << 15, 1 << 16, 1),   # W2 of 4 GB
    ((1 << 20) + 1, 64, 64, 1),  # past the row limit
    (64, (1 << 18) + 64, 64, 1), # past the width limit
])
def test_sizes_the_plan_refuses(lib, M, H, F, act):
    with pytest.raises(B.Mlp2Error) as e:
        B.Plan(M, H, F, act)
    assert e.value.code == B.ERR_UNSUPPORTED


def test_a_grouped_batch_may_exceed_4gb_of_x(lib):
    # 2^20 rows x 4096: X is 8 GB, but Z of 8192 columns exceeds the cache, so
    # the plan runs row groups whose X slices stay far below 4 GB
    plan = B.Plan(1 << 20, 4096, 8192, 1)
    assert plan.info()["row_group"] > 0
    plan.close()


def test_chain_refuses_operands_of_4gb(lib):
    with pytest.raises(B.Mlp2Error) as e:
        B.ChainPlan(1 << 20, [4096, 128], 1)  # X of 8 GB
    assert e.value.code == B.ERR_UNSUPPORTED
    with pytest.raises(B.Mlp2Error) as e:
        B.ChainPlan(64, [1 << 16, 1 << 15], 1)  # a 4 GB weight
    assert e.value.code == B.ERR_UNSUPPORTED
