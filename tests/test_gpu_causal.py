"""GPU parity of the causal-mask path (M_ij = -inf for j > i, eq. 1) against
the float64 oracle with the same mask: every output element at small and
ragged sizes (tiles skipped above the diagonal, diagonal tiles masked per
element), both Pass 1 forms, both dtypes and head dims; and sampled rows plus
global identities at N = 16384, d = 128 and at the causal benchmark workload
(B=4, H=12, N=16384, d=64)."""
import numpy as np
import pytest
import torch

import oracle
from tests.parity_util import (TOL, check_identities, check_rows, nrel, oracle_full, run_gpu_path, say,
                               to_dev)
from workloads import NAMES, WORKLOADS, as_f64, make_inputs, workload_inputs

pytestmark = pytest.mark.gpu

OUTS = ("O", "L", "D", "dQ", "dK", "dV", "alpha", "E", "Qt", "dOt", "Kt", "Vt")

CASES = [
    # B, H, N, d, dtype, seed, use_dq
    (1, 1, 256, 64, "f32", 60, True),
    (1, 2, 1, 64, "f32", 61, True),
    (1, 1, 31, 128, "f32", 62, False),
    (2, 1, 300, 128, "f32", 63, True),
    (1, 1, 65, 64, "bf16", 64, True),
    (2, 2, 257, 64, "bf16", 65, False),
    (1, 1, 1000, 128, "bf16", 66, True),
    (1, 3, 513, 128, "bf16", 67, False),
    (1, 1, 2048, 64, "bf16", 68, True),
]


def case_id(c):
    return f"B{c[0]}H{c[1]}N{c[2]}d{c[3]}{c[4]}s{c[5]}{'dq' if c[6] else 'six'}"


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_causal_full_path_matches_oracle(case):
    B, H, N, d, dt, seed, use_dq = case
    say(f"[causal] full path {case_id(case)}")
    x = make_inputs(B, H, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle_full(x, scale, causal=True)
    out = run_gpu_path(to_dev(x), scale, use_dq=use_dq, causal=True)
    errs = {}
    for k in OUTS:
        a, b = as_f64(out[k]), ref[k]
        if N == 1 and k in ("Qt", "Kt", "Vt", "dQ", "dK"):
            errs[k] = float(np.abs(a).max())           # exactly zero in exact arithmetic
        else:
            errs[k] = nrel(a, b)
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)


def test_causal_n16384_d128_sampled_rows_and_identities():
    w = WORKLOADS["bf16_b1h16_n16384_d128"]
    say(f"[causal] {w.name} under the causal mask: GPU path")
    x = workload_inputs(w)
    xd = to_dev(x)
    out = run_gpu_path(xd, w.scale, causal=True)
    check_rows(x, out, w, rows_per_head=32, seed=5005, causal=True)
    check_identities(xd, out)


@pytest.mark.parametrize("name", ["causal_bf16_b4h12_n16384_d64"])
def test_causal_paper_shape_sampled_rows_and_identities(name):
    """The causal benchmark workload (the paper's kernel shape), in the launch
    configuration the benchmark times."""
    w = WORKLOADS[name]
    say(f"[causal] {w.name}: GPU path")
    x = workload_inputs(w)
    xd = to_dev(x)
    out = run_gpu_path(xd, w.scale, causal=True)
    check_rows(x, out, w, rows_per_head=8, seed=5006, causal=True)
    check_identities(xd, out)
