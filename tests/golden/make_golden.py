"""Writes oracle_regression.json: frozen oracle outputs on tiny seeded inputs.

Calls only the oracle and the seeded input generator; run from the repo root:
    python tests/golden/make_golden.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import mlp2_oracle as O  # noqa: E402
from paper_2607_07862_amd import inputs as I  # noqa: E402

cases = []
for (M, H, F, act, seed) in [(2, 4, 6, 0, 100), (3, 8, 4, 1, 101), (2, 6, 5, 2, 102)]:
    d = I.make_inputs(M, H, F, act, seed)
    Y = O.mlp2(I.bits(d["X"]), I.bits(d["W1"]), I.bits(d["W2"]), M, H, F, act)
    cases.append({"M": M, "H": H, "F": F, "act": act, "seed": seed, "Y": [float(v) for v in Y.ravel()]})
out = {"about": "oracle outputs on seeded tiny inputs; regression fixture only (the pins are in test_oracle.py)",
       "cases": cases}
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_regression.json"), "w") as f:
    json.dump(out, f, indent=1)
print("wrote", len(cases), "cases")
