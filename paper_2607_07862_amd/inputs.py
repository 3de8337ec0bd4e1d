"""Seeded synthetic inputs for the two-layer MLP ``Y = act(X @ W1) @ W2``.

This module is shared by the tests, the bench and the smoke check.  It holds
none of the method's arithmetic: it only draws Gaussian numbers, scales them by
the initialisation's standard deviation and rounds them to bf16.  The oracle
and the HIP path both consume its output; neither is imported here.

Recipe (one per workload):
  * ``torch.Generator('cpu').manual_seed(seed)``;
  * fp32 ``randn`` drawn in the order X, W1 (for the gated MLP: Wg then Wu),
    W2;
  * X ~ N(0, 1); every weight ~ N(0, 1/fan_in) with the *standard deviation*
    equal to ``1/sqrt(fan_in)`` (fan_in = H for W1/Wg/Wu, F for W2), so the
    pre-activations are roughly N(0, 1);
  * scaled in fp32, then rounded to bf16 (round to nearest even).

Layouts (row-major, bf16): X [M, H]; W1 [H, F], or for the gated MLP the
packed ``[2, H, F]`` tensor holding Wg then Wu; W2 [F, H]; Y [M, H].

The workloads are shaped like LLM MLP layers (Llama-8B: H=4096, F=14336;
a 70B model: H=8192, F=28672; one tensor-parallel 1/8 shard: F=3584) plus a
tiny case; the paper's method is evaluated on such MLP layers (Sec. IV,
two-layer GEMM standing for the MLP).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

ACT_IDENTITY = 0
ACT_GELU_TANH = 1
ACT_SWIGLU = 2
ACT_NAMES = {"identity": ACT_IDENTITY, "gelu_tanh": ACT_GELU_TANH, "swiglu": ACT_SWIGLU}


@dataclass(frozen=True)
class Workload:
    name: str
    M: int
    H: int
    F: int
    act: int
    seed: int

    @property
    def gated(self) -> bool:
        return self.act == ACT_SWIGLU

    def weight_bytes(self) -> int:
        n1 = (2 if self.gated else 1) * self.H * self.F
        return 2 * (n1 + self.F * self.H)

    def alg_bytes(self) -> int:
        """HBM bytes the operation must move at least once: X, W1 (or Wg+Wu), W2, Y."""
        return self.weight_bytes() + 2 * (self.M * self.H) * 2

    def alg_flops(self) -> int:
        n_gemm1 = 2 if self.gated else 1
        return 2 * self.M * self.H * self.F * (n_gemm1 + 1)

    def z_bytes(self) -> int:
        return 2 * self.M * self.F


# The five MLP workloads (sizes, activation, seed).
WORKLOADS = {
    "tiny": Workload("tiny-64x512x2048-identity", 64, 512, 2048, ACT_IDENTITY, 0),
    "l8b_decode": Workload("llama8b-decode-128x4096x14336-gelu", 128, 4096, 14336, ACT_GELU_TANH, 1),
    "l8b_prefill": Workload("llama8b-prefill-2048x4096x14336-gelu", 2048, 4096, 14336, ACT_GELU_TANH, 2),
    "l70b_gated": Workload("llama70b-gated-256x8192x28672-swiglu", 256, 8192, 28672, ACT_SWIGLU, 3),
    "l70b_shard8": Workload("llama70b-tp8shard-32x8192x3584-gelu", 32, 8192, 3584, ACT_GELU_TANH, 4),
}
WORKLOAD_ORDER = ["tiny", "l8b_decode", "l8b_prefill", "l70b_gated", "l70b_shard8"]

# The paper's own workload (Sec. IV): Y = X A B with both weight matrices
# fixed at 8192 x 8192, no activation between the layers, and the row count
# of X swept over 1024 ... 32768.  A shape study beside the five workloads.
PAPER_ORDER = []
for _i, _m in enumerate((1024, 2048, 4096, 8192, 16384, 32768)):
    WORKLOADS[f"paper_m{_m}"] = Workload(f"paper-{_m}x8192x8192-identity", _m, 8192, 8192, ACT_IDENTITY, 10 + _i)
    PAPER_ORDER.append(f"paper_m{_m}")


def _randn_bf16(gen: torch.Generator, shape, std: float) -> torch.Tensor:
    t = torch.randn(*shape, generator=gen, dtype=torch.float32)
    if std != 1.0:
        t = t * torch.tensor(std, dtype=torch.float32)
    return t.to(torch.bfloat16)


def make_inputs(M: int, H: int, F: int, act: int, seed: int) -> dict:
    """Return CPU bf16 tensors ``X [M,H]``, ``W1 [H,F]`` (gated: ``[2,H,F]``), ``W2 [F,H]``."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(int(seed))
    X = _randn_bf16(gen, (M, H), 1.0)
    s1 = float(1.0 / np.sqrt(H))
    if act == ACT_SWIGLU:
        Wg = _randn_bf16(gen, (H, F), s1)
        Wu = _randn_bf16(gen, (H, F), s1)
        W1 = torch.stack([Wg, Wu], dim=0).contiguous()
    else:
        W1 = _randn_bf16(gen, (H, F), s1)
    W2 = _randn_bf16(gen, (F, H), float(1.0 / np.sqrt(F)))
    return {"X": X, "W1": W1, "W2": W2}


def chain_inputs(M: int, dims, seed: int) -> dict:
    """CPU bf16 tensors of a GEMM chain: ``X [M, D_0]`` ~ N(0, 1) and ``Ws``, one
    ``[D_{l-1}, D_l]`` per layer ~ N(0, 1/D_{l-1}) (the fan-in scaling of the workloads)."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(int(seed))
    X = _randn_bf16(gen, (M, dims[0]), 1.0)
    Ws = [_randn_bf16(gen, (dims[l], dims[l + 1]), float(1.0 / np.sqrt(dims[l]))) for l in range(len(dims) - 1)]
    return {"X": X, "Ws": Ws}


def workload_inputs(w: Workload) -> dict:
    return make_inputs(w.M, w.H, w.F, w.act, w.seed)


def bits(t: torch.Tensor) -> np.ndarray:
    """The raw bf16 bit patterns of a CPU bf16 tensor as a numpy uint16 array (no copy of values)."""
    assert t.dtype == torch.bfloat16 and t.device.type == "cpu"
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def from_bits(b: np.ndarray) -> torch.Tensor:
    """A CPU bf16 tensor holding the given uint16 bit patterns."""
    return torch.from_numpy(np.ascontiguousarray(b, dtype=np.uint16).view(np.int16)).view(torch.bfloat16)


def sample_rows(M: int, count: int, seed: int) -> np.ndarray:
    """A sorted, seeded sample of distinct row indexes that always includes the first and last rows."""
    if count >= M:
        return np.arange(M)
    rng = np.random.default_rng(1000 + seed)
    mid = rng.choice(np.arange(1, M - 1), size=max(count - 2, 0), replace=False)
    return np.unique(np.concatenate([[0, M - 1], mid]))


def sample_rows_per_block(M: int, block: int, count: int, seed: int) -> np.ndarray:
    """``sample_rows(M, count, seed)`` plus one seeded row inside every block of
    ``block`` consecutive rows (a different offset in each block), sorted."""
    rng = np.random.default_rng(2000 + seed)
    starts = np.arange(0, M, block)
    per = np.array([s + rng.integers(0, min(block, M - s)) for s in starts], dtype=np.int64)
    return np.unique(np.concatenate([sample_rows(M, count, seed), per]))
