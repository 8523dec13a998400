"""Writes tests/golden/bob_tiny_n5_d3.json from the float64 oracle only.

The paper prints no numeric worked example, so this fixture is not a
published value: it freezes the oracle's output on one tiny seeded case
(N=5, d=3, tau=1/sqrt(3), inputs from the shared generator with seed 2024,
float32) so that any later change to the oracle's arithmetic shows up as a
diff.  Run:  python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from workloads import as_f64, make_inputs  # noqa: E402


def main():
    x = make_inputs(1, 1, 5, 3, "f32", seed=2024)
    args = [as_f64(x[n])[0, 0] for n in ("Q", "K", "V", "dO", "UQ", "UK", "UV")]
    tau = 1 / np.sqrt(3)
    out = oracle.bob_head(*args, tau)
    doc = {
        "about": "Oracle BoB outputs for one tiny seeded head; eqs. 6-7 of the paper. "
                 "Not a paper-printed value (the paper prints none).",
        "N": 5, "d": 3, "tau": tau, "seed": 2024,
        "inputs": {n: a.tolist() for n, a in zip(("Q", "K", "V", "dO", "UQ", "UK", "UV"), args)},
        "outputs": {k: np.asarray(out[k]).tolist() for k in ("Qt", "Kt", "Vt", "dOt", "alpha", "E", "L", "D")},
    }
    with open(os.path.join(HERE, "bob_tiny_n5_d3.json"), "w") as f:
        json.dump(doc, f, indent=1)


if __name__ == "__main__":
    main()
