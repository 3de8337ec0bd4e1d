"""Helpers shared by the GPU tests: seeded inputs on the device, runs of both
modes through the C ABI, and comparison with the oracle."""
from __future__ import annotations

import numpy as np
import torch

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

# Statistical bar beside the elementwise bound: the relative RMS error of Y.
# bf16 rounding of Z and of Y each contribute about 2^-9/sqrt(3) ~ 0.11 % of
# the RMS of Y, so ~0.16 % is expected; 1 % leaves a 6x margin yet fails a
# single dropped K-slice out of 100 (~10 %).
REL_RMS_MAX = 1e-2


def device_inputs(d: dict) -> dict:
    return {k: v.to("cuda") for k, v in d.items()}


def run(plan: B.Plan, g: dict, mode: int, Y=None, stream=None):
    if Y is None:
        Y = torch.empty(plan.M, plan.H, dtype=torch.bfloat16, device="cuda")
    plan.run(g["X"], g["W1"], g["W2"], Y, mode, stream=stream)
    return Y


def workqueue_mode(plan: B.Plan, g: dict):
    """Y and Z of a workqueue-mode run (synchronised)."""
    Yq = run(plan, g, B.MODE_WORKQUEUE)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    return Yq, plan.intermediate()


def sentinel_mode(plan: B.Plan, g: dict):
    """Y of a sentinel-mode run (synchronised)."""
    Yn = run(plan, g, B.MODE_SENTINEL)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    return Yn


def both_modes(plan: B.Plan, g: dict):
    """Y and Z of a sequential run and of a pipelined run (each synchronised)."""
    Ys = run(plan, g, B.MODE_SEQUENTIAL)
    torch.cuda.synchronize()
    Zs = plan.intermediate()
    Yp = run(plan, g, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    Zp = plan.intermediate()
    assert plan.check() == B.OK
    return Ys, Zs, Yp, Zp


def bits_of(t: torch.Tensor) -> np.ndarray:
    return I.bits(t.detach().to("cpu"))


def assert_bit_equal(a: torch.Tensor, b: torch.Tensor, what: str):
    ba, bb = bits_of(a), bits_of(b)
    n = int(np.count_nonzero(ba != bb))
    assert n == 0, f"{what}: {n} of {ba.size} elements differ bitwise"


def assert_matches_oracle(Y: torch.Tensor, ref: np.ndarray, what: str):
    r = O.check_against(bits_of(Y), ref)
    assert r["ok"], f"{what}: {r['n_bad']} elements over the bound {r['bound']:.4g} (max err {r['max_abs_err']:.4g})"
    assert r["rel_rms"] <= REL_RMS_MAX, f"{what}: relative RMS error {r['rel_rms']:.3g}"
    return r
