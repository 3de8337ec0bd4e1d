"""Seeded random shapes through the default plan, on the GPU through the C ABI.

The hand-picked cases of the parity tests pin each tile shape; these draw the
sizes instead (a fixed seed, so every run tests the same shapes): ragged row
counts from 1 to about 1100, H and F any multiples of 64 up to 1536 and 3072
(odd ratios between them included), every activation.  Whatever tiles,
split-K and orders the plan picks, every mode gives the sequential mode's
bits on Y (and the one-launch modes on Z), and Y and Z match the fp64 oracle
within the elementwise bound.  GEMM chains likewise: one to four layers of
widths that differ from layer to layer, both modes bit-equal, Y within the
chain oracle's bound.
"""
import random

import pytest

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import binding as B
from paper_2607_07862_amd import inputs as I

from _gpu import assert_bit_equal, assert_matches_oracle, both_modes, device_inputs, sentinel_mode, workqueue_mode

pytestmark = pytest.mark.gpu


def _cases(n, seed):
    rng = random.Random(seed)
    out = []
    for _ in range(n):
        M = rng.choice([rng.randint(1, 64), rng.randint(65, 300), rng.randint(301, 1100)])
        out.append((M, 64 * rng.randint(1, 24), 64 * rng.randint(1, 48), rng.randrange(3)))
    return out


CASES = _cases(24, 20261202)


@pytest.mark.parametrize("M,H,F,act", CASES, ids=[f"{c[0]}x{c[1]}x{c[2]}-a{c[3]}" for c in CASES])
def test_random_shapes_every_mode(lib, M, H, F, act):
    print(f"\n[random shape] M={M} H={H} F={F} act={act}", flush=True)
    d = I.make_inputs(M, H, F, act, seed=M + 3 * H + 5 * F + act)
    g = device_inputs(d)
    plan = B.Plan(M, H, F, act)
    Ys, Zs, Yp, Zp = both_modes(plan, g)
    Yq, Zq = workqueue_mode(plan, g)
    Yn = sentinel_mode(plan, g)
    assert_bit_equal(Ys, Yp, "Y sequential vs pipelined")
    assert_bit_equal(Zs, Zp, "Z sequential vs pipelined")
    assert_bit_equal(Ys, Yq, "Y sequential vs workqueue")
    assert_bit_equal(Zs, Zq, "Z sequential vs workqueue")
    assert_bit_equal(Ys, Yn, "Y sequential vs sentinel")
    ref = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    assert_matches_oracle(Yp, ref, "Y")
    zref = O.intermediate(I.bits(d["X"]), I.bits(d["W1"]), M, H, F, act)
    assert_matches_oracle(Zp[:M], zref, "Z")
    plan.close()


def _chain_cases(n, seed):
    rng = random.Random(seed)
    out = []
    for _ in range(n):
        L = rng.randint(1, 4)
        M = rng.choice([rng.randint(1, 128), rng.randint(129, 700)])
        out.append((M, [128 * rng.randint(1, 12) for _ in range(L + 1)], rng.randrange(2)))
    return out


CHAIN_CASES = _chain_cases(12, 20261203)


@pytest.mark.parametrize("M,dims,act", CHAIN_CASES, ids=[f"{c[0]}x{'-'.join(map(str, c[1]))}-a{c[2]}" for c in CHAIN_CASES])
def test_random_chains_both_modes(lib, M, dims, act):
    import torch

    print(f"\n[random chain] M={M} dims={dims} act={act}", flush=True)
    d = I.chain_inputs(M, dims, seed=M + sum(dims) + act)
    X, Ws = d["X"].to("cuda"), [w.to("cuda") for w in d["Ws"]]
    plan = B.ChainPlan(M, dims, act)
    Ys = torch.empty(M, dims[-1], dtype=torch.bfloat16, device="cuda")
    Yp = torch.empty_like(Ys)
    plan.run(X, Ws, Ys, B.MODE_SEQUENTIAL)
    plan.run(X, Ws, Yp, B.MODE_TILE_PIPELINED)
    torch.cuda.synchronize()
    assert plan.check() == B.OK
    assert_bit_equal(Ys, Yp, "chain Y sequential vs pipelined")
    ref = O.chain(I.bits(d["X"]), [I.bits(w) for w in d["Ws"]], M, dims, act)
    assert_matches_oracle(Yp, ref, "chain Y")
    plan.close()
