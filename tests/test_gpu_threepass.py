"""GPU parity of the three-pass control schedule (App. "Three-pass versus
two-pass"): sweep 1 (alpha alone), sweep 2 (Qt, dOt, E with alpha given),
sweep 3 (the shared column pass) against the float64 oracle, every output
element at small and ragged sizes, dense and causal; and, at B=1 H=16
N=16384 d=128, sampled rows against the oracle plus agreement with the
two-pass outputs of the same inputs."""
import numpy as np
import pytest
import torch

from tests.parity_util import TOL, check_rows, nrel, oracle_full, say, to_dev
from workloads import NAMES, WORKLOADS, as_f64, make_inputs, workload_inputs

pytestmark = pytest.mark.gpu

OUTS = ("alpha", "E", "Qt", "dOt", "Kt", "Vt")

CASES = [
    # B, H, N, d, dtype, seed, causal
    (1, 1, 256, 64, "f32", 70, False),
    (2, 1, 77, 128, "f32", 71, True),
    (1, 1, 1, 64, "f32", 72, False),
    (1, 2, 300, 64, "bf16", 73, False),
    (1, 1, 513, 128, "bf16", 74, True),
    (2, 2, 1000, 128, "bf16", 75, False),
]


def case_id(c):
    return f"B{c[0]}H{c[1]}N{c[2]}d{c[3]}{c[4]}{'causal' if c[6] else ''}"


def run3(xd, scale, causal):
    import paper_2609_24089_amd as fb
    fb.load_library()
    out = fb.bob3(*[xd[n] for n in NAMES], scale, causal=causal)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_threepass_matches_oracle(case):
    B, H, N, d, dt, seed, causal = case
    say(f"[3pass] {case_id(case)}")
    x = make_inputs(B, H, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle_full(x, scale, causal=causal)
    out = run3(to_dev(x), scale, causal)
    errs = {}
    for k in OUTS:
        a = as_f64(out[k])
        if N == 1 and k in ("Qt", "Kt", "Vt"):
            errs[k] = float(np.abs(a).max())           # exactly zero in exact arithmetic
        else:
            errs[k] = nrel(a, ref[k])
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)


def test_threepass_n16384_d128_rows_and_agreement_with_two_pass():
    import paper_2609_24089_amd as fb
    w = WORKLOADS["bf16_b1h16_n16384_d128"]
    say(f"[3pass] {w.name}")
    x = workload_inputs(w)
    xd = to_dev(x)
    out3 = run3(xd, w.scale, False)
    check_rows(x, out3, w, rows_per_head=32, seed=7010, keys=("Qt", "dOt", "alpha", "E"))
    out2 = fb.bob(*[xd[n] for n in NAMES], w.scale)
    torch.cuda.synchronize()
    diffs = {k: nrel(as_f64(out3[k]), as_f64(out2[k])) for k in OUTS}
    say("   three-pass vs two-pass", {k: f"{v:.2e}" for k, v in diffs.items()})
    for k, e in diffs.items():
        assert e <= TOL["bf16"], (k, e)
