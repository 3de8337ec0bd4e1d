"""CPU oracle for the two-layer MLP (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never calls it and must fail loudly when its compiled
extension is missing.
"""
from .mlp2_oracle import (  # noqa: F401
    ACT_GELU_TANH,
    ACT_IDENTITY,
    ACT_SWIGLU,
    bf16_bits_to_f64,
    check_against,
    gelu_tanh,
    intermediate,
    mlp2,
    silu,
    tolerance_bound,
)
