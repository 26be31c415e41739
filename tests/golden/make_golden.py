"""Writes ``dense784x100_seed0.json``: the oracle's fp32 training step on the
single-layer workload (x[100,784] ~ U(0,1), W[784,100] ~ N(0, 0.1), b = 0,
L = 1/2 sum h^2, lr = 0.01; the example of the paper's Figure 1 in
batch-major form), as a regression anchor for the oracle.

The paper prints no numeric worked example, so every value here comes from
the oracle itself; this script calls only ``oracle`` and the seeded input
generator. Run from the repository root: ``python tests/golden/make_golden.py``.
"""

import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_1603_04467_amd import workloads  # noqa: E402

ROWS = [0, 17, 99]
COLS = [0, 5, 99]


def compute():
    w = workloads.workload("dense784x100")
    inp = workloads.generate(w, seed=0)
    x = inp["x"].astype(np.float64)
    W = inp["weights"][0].astype(np.float64)
    b = inp["biases"][0].astype(np.float64)
    out = oracle.dense_step(x, [W], [b], [True], act="f32", lr=w.lr)
    h = out["h"][1]
    return {
        "workload": w.name,
        "seed": 0,
        "loss": out["loss"],
        "relu_active": int(np.count_nonzero(h)),
        "h": [[float(h[i, j]) for j in COLS] for i in ROWS],
        "db": [float(out["db"][0][j]) for j in COLS],
        "dw": [[float(out["dw"][0][i, j]) for j in COLS] for i in [0, 400, 783]],
        "dx": [[float(out["dx"][0][i, j]) for j in [0, 400, 783]] for i in ROWS],
        "new_w": [[float(out["new_weights"][0][i, j]) for j in COLS] for i in [0, 400, 783]],
    }


if __name__ == "__main__":
    with open(os.path.join(HERE, "dense784x100_seed0.json"), "w") as f:
        json.dump(compute(), f, indent=1)
        f.write("\n")
