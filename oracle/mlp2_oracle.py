"""fp64 CPU oracle for ``Y = act(X @ W1) @ W2`` from bf16 inputs.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py``'s ``cpu_baseline`` leg may import or run this module.  It shares
no code with the HIP path (no kernels, headers, helpers or tables) and never
imports it.

What it computes (CTA-pipelining, arXiv 2607.07862):
  * Sec. IV states the workload: the two-layer GEMM ``Y = X A B`` stands for
    an LLM MLP layer, with X the activations and A, B the weights; inputs
    and outputs are bf16 with fp32 accumulation (Sec. III-C and Sec. IV).
  * Pipelining (Sec. III-A) only changes *when* a consumer tile runs, never
    the arithmetic: a consumer tile starts once every producer tile it reads
    is complete.  The method therefore reaches exactly the plain definition
    of the two-layer product, which is what this oracle writes out.
  * The paper leaves the activation out of its workload (Sec. IV); the workloads
    built here put one back between the GEMMs: identity, GELU with the tanh
    approximation, or SwiGLU ``silu(X Wg) * (X Wu)`` with the packed weight
    ``W1 = [Wg; Wu]`` of shape ``[2, H, F]``.

Readings where the paper is silent (each listed in the design notes):
  * the intermediate Z is kept in fp64 here (the plain definition); the GPU
    path stores it as bf16, which the tolerance absorbs;
  * GELU is the tanh form ``0.5 p (1 + tanh(sqrt(2/pi) (p + 0.044715 p^3)))``;
  * SiLU is applied to the Wg branch.

Every step is fp64: bf16 inputs decode exactly to fp64; products of two bf16
values are exact in fp64; the only rounding is in the fp64 sums (matmul, a
library primitive used as one step) and in ``tanh``/``exp``.
"""
from __future__ import annotations

import numpy as np

ACT_IDENTITY = 0
ACT_GELU_TANH = 1
ACT_SWIGLU = 2

# Elementwise acceptance bound for a bf16 result Y against the fp64 reference:
# |Y - Y_ref| <= REL_OF_MAX * max|Y_ref| + ABS_FLOOR, with max over the tensor.
REL_OF_MAX = 2e-2
ABS_FLOOR = 1e-3


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) exactly: the bf16 value is the fp32 with these 16 high bits."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def gelu_tanh(p: np.ndarray) -> np.ndarray:
    """GELU, tanh approximation: 0.5 p (1 + tanh(sqrt(2/pi) (p + 0.044715 p^3)))."""
    c = np.sqrt(2.0 / np.pi)
    return 0.5 * p * (1.0 + np.tanh(c * (p + 0.044715 * p * p * p)))


def silu(g: np.ndarray) -> np.ndarray:
    """SiLU: g * sigmoid(g) = g / (1 + exp(-g))."""
    return g / (1.0 + np.exp(-g))


def _check_shapes(X, W1, W2, M, H, F, act):
    if act not in (ACT_IDENTITY, ACT_GELU_TANH, ACT_SWIGLU):
        raise ValueError(f"unknown activation {act}")
    n1 = 2 if act == ACT_SWIGLU else 1
    if X.size != M * H:
        raise ValueError("X must hold M*H elements")
    if W1.size != n1 * H * F:
        raise ValueError("W1 must hold H*F elements (2*H*F for SwiGLU)")
    if W2 is not None and W2.size != F * H:
        raise ValueError("W2 must hold F*H elements")


def intermediate(X_bits, W1_bits, M: int, H: int, F: int, act: int, rows=None) -> np.ndarray:
    """The first layer Z = act(X @ W1) in fp64, for all rows or the given row indexes.

    X_bits [M,H] and W1_bits [H,F] (SwiGLU: [2,H,F], Wg then Wu) are bf16 bit patterns.
    """
    _check_shapes(X_bits, W1_bits, None, M, H, F, act)
    X = bf16_bits_to_f64(X_bits).reshape(M, H)
    if rows is not None:
        X = X[np.asarray(rows, dtype=np.int64)]
    if act == ACT_SWIGLU:
        W = bf16_bits_to_f64(W1_bits).reshape(2, H, F)
        G = X @ W[0]
        U = X @ W[1]
        return silu(G) * U
    W = bf16_bits_to_f64(W1_bits).reshape(H, F)
    P = X @ W
    if act == ACT_GELU_TANH:
        return gelu_tanh(P)
    return P


def mlp2(X_bits, W1_bits, W2_bits, M: int, H: int, F: int, act: int, rows=None) -> np.ndarray:
    """Y = act(X @ W1) @ W2 in fp64 (rows: optional subset of output rows). Returns [rows, H]."""
    _check_shapes(X_bits, W1_bits, W2_bits, M, H, F, act)
    Z = intermediate(X_bits, W1_bits, M, H, F, act, rows)
    W2 = bf16_bits_to_f64(W2_bits).reshape(F, H)
    return Z @ W2


def chain(X_bits, W_bits: list, M: int, dims: list, act: int, rows=None) -> np.ndarray:
    """An L-layer GEMM chain in fp64: Z_0 = X, Z_l = act(Z_{l-1} @ W_l) for
    l < L and Y = Z_{L-1} @ W_L (rows: optional subset of output rows).

    The paper's pipelining carries over to a chain of GEMMs whose middle
    kernels both consume the previous output and produce the next (Sec.
    III-A, the producer/consumer relation applied at every boundary); as for
    two layers it changes only when a tile runs, so the result is the plain
    product, with the activation after every layer but the last (identity or
    GELU, tanh form).  dims = [D_0, ..., D_L]: X is [M, D_0], W_l is
    [D_{l-1}, D_l] (bf16 bit patterns); the intermediates stay fp64.
    """
    L = len(W_bits)
    if L < 1 or len(dims) != L + 1 or act not in (ACT_IDENTITY, ACT_GELU_TANH):
        raise ValueError("chain: need L >= 1 weights, L + 1 widths and an identity or GELU activation")
    if np.asarray(X_bits).size != M * dims[0]:
        raise ValueError("chain: X size does not match M x D_0")
    Z = bf16_bits_to_f64(X_bits).reshape(M, dims[0])
    if rows is not None:
        Z = Z[np.asarray(rows, dtype=np.int64)]
    for l, Wb in enumerate(W_bits):
        if np.asarray(Wb).size != dims[l] * dims[l + 1]:
            raise ValueError(f"chain: W_{l + 1} size does not match D_{l} x D_{l + 1}")
        Z = Z @ bf16_bits_to_f64(Wb).reshape(dims[l], dims[l + 1])
        if l < L - 1 and act == ACT_GELU_TANH:
            Z = gelu_tanh(Z)
    return Z


def tolerance_bound(Y_ref: np.ndarray) -> float:
    """The elementwise acceptance bound REL_OF_MAX * max|Y_ref| + ABS_FLOOR."""
    m = float(np.max(np.abs(Y_ref))) if Y_ref.size else 0.0
    return REL_OF_MAX * m + ABS_FLOOR


def check_against(Y_bits, Y_ref: np.ndarray) -> dict:
    """Compare a bf16 result (bit patterns) with the fp64 reference.

    Returns ``ok`` (every element within ``tolerance_bound``), the bound, the
    largest absolute error, the relative RMS error ``||Y-Y_ref|| / ||Y_ref||``
    and the count of elements over the bound.  Non-finite values fail.
    """
    Y = bf16_bits_to_f64(Y_bits).reshape(Y_ref.shape)
    bound = tolerance_bound(Y_ref)
    if Y.size == 0:
        return {"ok": True, "bound": bound, "max_abs_err": 0.0, "rel_rms": 0.0, "n_bad": 0, "ref_max": 0.0}
    err = np.abs(Y - Y_ref)
    finite = np.isfinite(Y)
    n_bad = int(np.count_nonzero(~finite) + np.count_nonzero(err[finite] > bound))
    den = float(np.sqrt(np.sum(Y_ref * Y_ref)))
    rel_rms = float(np.sqrt(np.sum(np.where(finite, err, 0.0) ** 2)) / den) if den > 0 else float(np.max(err))
    return {
        "ok": n_bad == 0,
        "bound": bound,
        "max_abs_err": float(np.max(np.where(finite, err, np.inf))),
        "rel_rms": rel_rms,
        "n_bad": n_bad,
        "ref_max": float(np.max(np.abs(Y_ref))),
    }
