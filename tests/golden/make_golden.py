"""Writes tests/golden/tiny_filter_4x8.json from the float64 oracle only.

A regression fixture: a 1 x 4 x 8 token grid with 8 channels in 2 blocks of 4, weights
N(0, 0.3^2), lambda 0.05, keep 1.0, seed 7.  It guards the oracle against silent
drift; the pins in tests/test_oracle_pins.py are what tie it to the paper.
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
import oracle  # noqa: E402

if __name__ == "__main__":
    rng = np.random.default_rng(7)
    nb, bs = 2, 4
    inputs = {
        "x": rng.standard_normal((1, 4, 8, nb * bs)),
        "w1": 0.3 * rng.standard_normal((nb, bs, bs, 2)),
        "b1": 0.3 * rng.standard_normal((nb, bs, 2)),
        "w2": 0.3 * rng.standard_normal((nb, bs, bs, 2)),
        "b2": 0.3 * rng.standard_normal((nb, bs, 2)),
    }
    lam, keep = 0.05, 1.0
    out = oracle.filter_forward(inputs["x"], inputs["w1"], inputs["b1"], inputs["w2"],
                                inputs["b2"], nb, lam, keep)
    doc = {"source": "tests/golden/make_golden.py (oracle only)", "num_blocks": nb, "lam": lam,
           "keep": keep, "inputs": {k: v.tolist() for k, v in inputs.items()},
           "out": out.tolist()}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_filter_4x8.json")
    with open(path, "w") as f:
        json.dump(doc, f)
    print(path)
