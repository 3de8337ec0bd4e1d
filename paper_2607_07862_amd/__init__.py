"""Tile-pipelined two-layer MLP ``Y = act(X @ W1) @ W2`` for AMD MI355X (gfx950).

The computation lives in the HIP library ``libmlp2.so`` (C ABI in
``include/mlp2.h``); ``binding`` marshals arguments to it through ctypes and
``inputs`` draws the seeded synthetic workloads.  Importing the package does
not load the library; ``binding.load()`` does, and raises if it is missing.
"""
__all__ = ["binding", "inputs", "build"]
