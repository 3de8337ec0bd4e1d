"""Pins of the oracle's GEMM chain (fp64, CPU only).

* exact rational loops over every layer on tiny chains (brute force);
* a two-layer chain is the pinned two-layer product, GELU included;
* identity activation: the chain equals X times the product of the weights
  (associativity, a different evaluation order);
* identity weights give the activation applied L - 1 times to X; zero
  weights give exactly zero; a row subset equals the same rows of the whole;
* a planted mistake (an activation on the last layer, a dropped layer) is
  caught by these checks.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import mlp2_oracle as O


def _bits(a: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of the fp32 values (round to nearest even)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _case(M, dims, seed):
    rng = np.random.default_rng(seed)
    X = _bits(rng.standard_normal((M, dims[0])))
    Ws = [_bits(rng.standard_normal((dims[l], dims[l + 1])) / np.sqrt(dims[l])) for l in range(len(dims) - 1)]
    return X, Ws


@pytest.mark.parametrize("M,dims,seed", [(1, [1, 1, 1, 1], 0), (2, [3, 2, 4, 3], 1), (3, [4, 5, 3, 2, 4], 2)])
def test_bruteforce_exact_rational_identity_chain(M, dims, seed):
    X, Ws = _case(M, dims, seed)
    Z = [[Fraction(float(v)) for v in row] for row in O.bf16_bits_to_f64(X).reshape(M, dims[0])]
    for l, Wb in enumerate(Ws):
        W = [[Fraction(float(v)) for v in row] for row in O.bf16_bits_to_f64(Wb).reshape(dims[l], dims[l + 1])]
        Z = [[sum(Z[m][k] * W[k][n] for k in range(dims[l])) for n in range(dims[l + 1])] for m in range(M)]
    got = O.chain(X, Ws, M, dims, O.ACT_IDENTITY)
    scale = max(1e-300, max(abs(float(v)) for row in Z for v in row))
    for m in range(M):
        for n in range(dims[-1]):
            assert abs(got[m, n] - float(Z[m][n])) <= 1e-13 * scale


@pytest.mark.parametrize("act", [O.ACT_IDENTITY, O.ACT_GELU_TANH])
def test_two_layers_are_the_pinned_product(act):
    M, H, F = 5, 8, 12
    X, (W1, W2) = _case(M, [H, F, H], 3)
    np.testing.assert_array_equal(O.chain(X, [W1, W2], M, [H, F, H], act), O.mlp2(X, W1, W2, M, H, F, act))


def test_identity_act_is_x_times_the_weight_product():
    M, dims = 4, [6, 10, 7, 9, 5]
    X, Ws = _case(M, dims, 4)
    P = np.eye(dims[0])
    for l, Wb in enumerate(Ws):
        P = P @ O.bf16_bits_to_f64(Wb).reshape(dims[l], dims[l + 1])
    want = O.bf16_bits_to_f64(X).reshape(M, dims[0]) @ P
    got = O.chain(X, Ws, M, dims, O.ACT_IDENTITY)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12 * np.max(np.abs(want)))


@pytest.mark.parametrize("L", [1, 3, 4])
def test_identity_weights_apply_the_activation_l_minus_1_times(L):
    M, D = 6, 8
    X, _ = _case(M, [D, D], 5)
    eye = _bits(np.eye(D))
    x = O.bf16_bits_to_f64(X).reshape(M, D)
    want = x
    for _ in range(L - 1):
        want = O.gelu_tanh(want)
    np.testing.assert_array_equal(O.chain(X, [eye] * L, M, [D] * (L + 1), O.ACT_GELU_TANH), want)


def test_zero_weights_give_zero_and_rows_match_the_whole():
    M, dims = 7, [8, 16, 8, 12]
    X, Ws = _case(M, dims, 6)
    zeros = [np.zeros_like(w) for w in Ws]
    assert np.all(O.chain(X, zeros, M, dims, O.ACT_GELU_TANH) == 0)
    full = O.chain(X, Ws, M, dims, O.ACT_GELU_TANH)
    rows = [0, 3, 6]
    np.testing.assert_array_equal(O.chain(X, Ws, M, dims, O.ACT_GELU_TANH, rows=rows), full[rows])


def test_planted_mistakes_are_caught():
    M, dims = 3, [4, 6, 6, 4]
    X, Ws = _case(M, dims, 7)
    good = O.chain(X, Ws, M, dims, O.ACT_GELU_TANH)
    # an activation after the last layer as well
    z = O.bf16_bits_to_f64(X).reshape(M, dims[0])
    for l, Wb in enumerate(Ws):
        z = O.gelu_tanh(z @ O.bf16_bits_to_f64(Wb).reshape(dims[l], dims[l + 1]))
    assert not np.allclose(z, good)
    # a dropped middle layer (square, so the shapes still fit)
    assert not np.allclose(O.chain(X, [Ws[0], Ws[2]], M, [4, 6, 4], O.ACT_GELU_TANH), good)
    with pytest.raises(ValueError):
        O.chain(X, Ws[:2], M, dims, O.ACT_GELU_TANH)
