"""Pins of the fp64 oracle against facts fixed outside it (no GPU needed).

Each test would fail under a plausible mistake in the oracle: a transposed
operand or wrong index (brute force on non-square shapes, the hand-worked
example), a dropped term (brute force, associativity), a wrong sign or
constant in an activation (library routines, symmetry invariants, the exact
erf form), the SwiGLU branch or packing order (the worked gated example).
"""
import json
import math
import os
from fractions import Fraction

import mpmath
import numpy as np
import pytest
import torch

from oracle import mlp2_oracle as O
from paper_2607_07862_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f2bits(a) -> np.ndarray:
    """Exact bf16 bit patterns of values that are already bf16-representable (asserted)."""
    t = torch.tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)
    back = t.to(torch.float32).numpy()
    assert np.array_equal(back, np.asarray(a, dtype=np.float32)), "value not exact in bf16"
    return I.bits(t)


def rand_case(M, H, F, act, seed):
    d = I.make_inputs(M, H, F, act, seed)
    return I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"])


# ---------------------------------------------------------------- decoding


def test_bf16_decode_exact_against_torch():
    g = torch.Generator().manual_seed(7)
    t = (torch.randn(4096, generator=g) * 37).to(torch.bfloat16)
    special = torch.tensor([0.0, -0.0, 1.0, -2.5, 3.0e38, 1e-40, float("inf")], dtype=torch.bfloat16)
    for x in (t, special):
        got = O.bf16_bits_to_f64(I.bits(x))
        want = x.to(torch.float64).numpy()
        assert np.array_equal(got, want)
    # sign of zero survives
    assert math.copysign(1.0, O.bf16_bits_to_f64(np.array([0x8000], np.uint16))[0]) == -1.0


# ---------------------------------------------------------------- worked examples


def test_worked_identity_example_exact():
    g = json.load(open(os.path.join(GOLDEN, "worked_identity.json")))
    X, W1, W2 = f2bits(g["X"]), f2bits(g["W1"]), f2bits(g["W2"])
    Z = O.intermediate(X, W1, g["M"], g["H"], g["F"], g["act"])
    Y = O.mlp2(X, W1, W2, g["M"], g["H"], g["F"], g["act"])
    assert np.array_equal(Z, np.array(g["Z"], dtype=np.float64))
    assert np.array_equal(Y, np.array(g["Y"], dtype=np.float64))


def test_worked_swiglu_example_branch_and_packing():
    g = json.load(open(os.path.join(GOLDEN, "worked_swiglu.json")))
    W1 = f2bits(np.stack([np.array(g["Wg"]), np.array(g["Wu"])]))
    Y = O.mlp2(f2bits(g["X"]), W1, f2bits(g["W2"]), g["M"], g["H"], g["F"], g["act"])
    want = np.array([[2.0 / (1.0 + math.exp(-1.0)), 2.0 / (1.0 + math.exp(1.0))]])
    assert np.allclose(Y, want, rtol=1e-15, atol=0)
    wrong = np.array([[2.0 / (1.0 + math.exp(-2.0)), 2.0 / (1.0 + math.exp(2.0))]])
    assert not np.allclose(Y, wrong, rtol=1e-3)


# ---------------------------------------------------------------- brute force


def _frac(bits):
    return [Fraction(float(v)) for v in O.bf16_bits_to_f64(bits).ravel()]


@pytest.mark.parametrize("M,H,F,seed", [(1, 1, 1, 0), (2, 3, 5, 1), (5, 4, 3, 2), (7, 8, 6, 3), (3, 8, 8, 4)])
def test_bruteforce_exact_rational_identity(M, H, F, seed):
    """Exact rational triple loops for Y = (X W1) W2; the oracle must agree to fp64 rounding."""
    X, W1, W2 = rand_case(M, H, F, O.ACT_IDENTITY, seed)
    x, w1, w2 = _frac(X), _frac(W1), _frac(W2)
    Z = [[sum(x[m * H + h] * w1[h * F + f] for h in range(H)) for f in range(F)] for m in range(M)]
    Y = [[sum(Z[m][f] * w2[f * H + n] for f in range(F)) for n in range(H)] for m in range(M)]
    got = O.mlp2(X, W1, W2, M, H, F, O.ACT_IDENTITY)
    scale = max(1e-300, max(abs(float(v)) for row in Y for v in row))
    for m in range(M):
        for n in range(H):
            assert abs(got[m, n] - float(Y[m][n])) <= 1e-14 * scale


def _mp_gelu(p):
    return mpmath.mpf("0.5") * p * (1 + mpmath.tanh(mpmath.sqrt(2 / mpmath.pi) * (p + mpmath.mpf("0.044715") * p**3)))


def _mp_silu(g):
    return g / (1 + mpmath.exp(-g))


@pytest.mark.parametrize("act", [O.ACT_GELU_TANH, O.ACT_SWIGLU])
@pytest.mark.parametrize("M,H,F,seed", [(2, 3, 5, 11), (4, 8, 6, 12), (3, 5, 8, 13)])
def test_bruteforce_high_precision_activations(act, M, H, F, seed):
    """40-digit loops; agreement to 1e-12 relative pins indexing, packing and the act's evaluation."""
    mpmath.mp.dps = 40
    X, W1, W2 = rand_case(M, H, F, act, seed)
    x = [mpmath.mpf(float(v)) for v in O.bf16_bits_to_f64(X).ravel()]
    w1 = [mpmath.mpf(float(v)) for v in O.bf16_bits_to_f64(W1).ravel()]
    w2 = [mpmath.mpf(float(v)) for v in O.bf16_bits_to_f64(W2).ravel()]
    Y = []
    for m in range(M):
        z = []
        for f in range(F):
            if act == O.ACT_SWIGLU:
                g = mpmath.fsum(x[m * H + h] * w1[h * F + f] for h in range(H))
                u = mpmath.fsum(x[m * H + h] * w1[H * F + h * F + f] for h in range(H))
                z.append(_mp_silu(g) * u)
            else:
                z.append(_mp_gelu(mpmath.fsum(x[m * H + h] * w1[h * F + f] for h in range(H))))
        Y.append([mpmath.fsum(z[f] * w2[f * H + n] for f in range(F)) for n in range(H)])
    got = O.mlp2(X, W1, W2, M, H, F, act)
    scale = max(abs(float(v)) for row in Y for v in row)
    for m in range(M):
        for n in range(H):
            assert abs(got[m, n] - float(Y[m][n])) <= 1e-12 * scale


# ---------------------------------------------------------------- activations vs library / closed forms


def test_gelu_tanh_matches_torch_library():
    p = np.linspace(-12, 12, 48001)
    ref = torch.nn.functional.gelu(torch.tensor(p, dtype=torch.float64), approximate="tanh").numpy()
    assert np.max(np.abs(O.gelu_tanh(p) - ref)) <= 1e-13


def test_silu_matches_torch_library():
    g = np.linspace(-40, 40, 48001)
    ref = torch.nn.functional.silu(torch.tensor(g, dtype=torch.float64)).numpy()
    assert np.max(np.abs(O.silu(g) - ref)) <= 1e-13


def test_activation_closed_forms_and_invariants():
    x = np.linspace(-9, 9, 18001)
    # act(x) - act(-x) = x holds exactly in real arithmetic for both x*sigmoid-type forms
    assert np.max(np.abs(O.gelu_tanh(x) - O.gelu_tanh(-x) - x)) <= 1e-14 * 10
    assert np.max(np.abs(O.silu(x) - O.silu(-x) - x)) <= 1e-14 * 10
    assert O.gelu_tanh(np.array([0.0]))[0] == 0.0 and O.silu(np.array([0.0]))[0] == 0.0
    # slopes at 0 are 1/2
    h = 1e-6
    assert abs((O.gelu_tanh(np.array([h]))[0] - O.gelu_tanh(np.array([-h]))[0]) / (2 * h) - 0.5) < 1e-9
    assert abs((O.silu(np.array([h]))[0] - O.silu(np.array([-h]))[0]) / (2 * h) - 0.5) < 1e-9
    # tails: gelu(x) -> x for large x, -> 0 for very negative x
    assert abs(O.gelu_tanh(np.array([30.0]))[0] - 30.0) < 1e-12
    assert abs(O.gelu_tanh(np.array([-30.0]))[0]) < 1e-12


def test_gelu_tanh_close_to_exact_erf_form():
    """The tanh form approximates x * Phi(x) to within 5e-4 everywhere (max deviation ~4.7e-4 near |x|=2.7)."""
    x = np.linspace(-10, 10, 40001)
    exact = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in x])
    dev = np.max(np.abs(O.gelu_tanh(x) - exact))
    assert 1e-4 < dev < 5e-4


# ---------------------------------------------------------------- structural cases


@pytest.mark.parametrize("act", [O.ACT_IDENTITY, O.ACT_GELU_TANH])
def test_identity_weights_give_act_of_x(act):
    M, H = 9, 16
    d = I.make_inputs(M, H, H, act, 21)
    X = I.bits(d["X"])
    eye = f2bits(np.eye(H))
    Y = O.mlp2(X, eye, eye, M, H, H, act)
    x = O.bf16_bits_to_f64(X).reshape(M, H)
    want = x if act == O.ACT_IDENTITY else O.gelu_tanh(x)
    assert np.array_equal(Y, want)


def test_identity_weights_swiglu():
    M, H = 5, 8
    X = I.bits(I.make_inputs(M, H, H, O.ACT_SWIGLU, 22)["X"])
    eye = np.eye(H)
    W1 = f2bits(np.stack([eye, 2 * eye]))
    Y = O.mlp2(X, W1, f2bits(eye), M, H, H, O.ACT_SWIGLU)
    x = O.bf16_bits_to_f64(X).reshape(M, H)
    assert np.allclose(Y, O.silu(x) * 2 * x, rtol=1e-15, atol=0)


@pytest.mark.parametrize("act", [O.ACT_IDENTITY, O.ACT_GELU_TANH, O.ACT_SWIGLU])
def test_zero_weights_give_zero(act):
    M, H, F = 6, 8, 12
    X = I.bits(I.make_inputs(M, H, F, act, 23)["X"])
    n1 = 2 if act == O.ACT_SWIGLU else 1
    Y = O.mlp2(X, np.zeros(n1 * H * F, np.uint16), np.zeros(F * H, np.uint16), M, H, F, act)
    assert np.all(Y == 0.0)
    # zero second layer alone
    d = I.make_inputs(M, H, F, act, 24)
    Y2 = O.mlp2(X, I.bits(d["W1"]), np.zeros(F * H, np.uint16), M, H, F, act)
    assert np.all(Y2 == 0.0)


def test_linearity_identity_act():
    """oracle(a X1 + b X2) = a oracle(X1) + b oracle(X2) with exact bf16 small-integer inputs."""
    M, H, F = 6, 16, 24
    rng = np.random.default_rng(5)
    X1 = rng.integers(-8, 9, size=(M, H)).astype(np.float64)
    X2 = rng.integers(-8, 9, size=(M, H)).astype(np.float64)
    d = I.make_inputs(M, H, F, O.ACT_IDENTITY, 25)
    W1, W2 = I.bits(d["W1"]), I.bits(d["W2"])
    a, b = 2.0, -0.5
    Ya = O.mlp2(f2bits(a * X1 + b * X2), W1, W2, M, H, F, 0)
    Yb = a * O.mlp2(f2bits(X1), W1, W2, M, H, F, 0) + b * O.mlp2(f2bits(X2), W1, W2, M, H, F, 0)
    assert np.max(np.abs(Ya - Yb)) <= 1e-12 * np.max(np.abs(Ya))


def test_associativity_identity_act():
    """(X W1) W2 = X (W1 W2): a different contraction order gives the same product."""
    M, H, F = 7, 48, 80
    X, W1, W2 = rand_case(M, H, F, O.ACT_IDENTITY, 26)
    Y = O.mlp2(X, W1, W2, M, H, F, 0)
    x = O.bf16_bits_to_f64(X).reshape(M, H)
    w1 = O.bf16_bits_to_f64(W1).reshape(H, F)
    w2 = O.bf16_bits_to_f64(W2).reshape(F, H)
    assert np.max(np.abs(Y - x @ (w1 @ w2))) <= 1e-12 * np.max(np.abs(Y))


def test_row_subset_matches_full():
    M, H, F = 33, 64, 96
    for act in (0, 1, 2):
        X, W1, W2 = rand_case(M, H, F, act, 27 + act)
        full = O.mlp2(X, W1, W2, M, H, F, act)
        rows = I.sample_rows(M, 5, 3)
        assert np.array_equal(O.mlp2(X, W1, W2, M, H, F, act, rows=rows), full[rows])


def test_shape_validation():
    with pytest.raises(ValueError):
        O.mlp2(np.zeros(4, np.uint16), np.zeros(4, np.uint16), np.zeros(4, np.uint16), 2, 2, 2, 7)
    with pytest.raises(ValueError):
        O.mlp2(np.zeros(3, np.uint16), np.zeros(4, np.uint16), np.zeros(4, np.uint16), 2, 2, 2, 0)
    with pytest.raises(ValueError):
        O.mlp2(np.zeros(4, np.uint16), np.zeros(4, np.uint16), np.zeros(4, np.uint16), 2, 2, 2, 2)


# ---------------------------------------------------------------- acceptance check


def test_check_against_detects_planted_errors():
    M, H, F = 8, 32, 64
    X, W1, W2 = rand_case(M, H, F, 1, 30)
    ref = O.mlp2(X, W1, W2, M, H, F, 1)
    y = I.bits(torch.tensor(ref, dtype=torch.float32).to(torch.bfloat16))
    r = O.check_against(y, ref)
    assert r["ok"] and r["rel_rms"] < 4e-3
    bad = y.copy().reshape(M, H)
    # push one element just over the bound
    v = float(O.bf16_bits_to_f64(bad[3:4, 5:6])[0, 0]) + 1.5 * r["bound"]
    bad[3, 5] = f2bits([np.float32(torch.tensor(v).to(torch.bfloat16).item())])[0]
    r2 = O.check_against(bad, ref)
    assert not r2["ok"] and r2["n_bad"] == 1
    nan = y.copy()
    nan[0] = 0x7FC0
    assert not O.check_against(nan, ref)["ok"]


def test_golden_regression_values():
    """Frozen oracle outputs written by tests/golden/make_golden.py (which calls only the oracle)."""
    g = json.load(open(os.path.join(GOLDEN, "oracle_regression.json")))
    for case in g["cases"]:
        X, W1, W2 = rand_case(case["M"], case["H"], case["F"], case["act"], case["seed"])
        Y = O.mlp2(X, W1, W2, case["M"], case["H"], case["F"], case["act"])
        assert np.allclose(Y.ravel(), np.array(case["Y"]), rtol=1e-13, atol=1e-15)
