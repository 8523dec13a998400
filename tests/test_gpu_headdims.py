"""GPU parity at head dims 32 and 256 (bf16; fp32 at d = 32): the whole
path (both Pass 1 forms) and the three-pass control schedule against the
float64 oracle, dense and causal, ragged N.  d = 32 uses the row-pair
interleaved LDS layout; d = 256 the d = 128 chunk order per 256-byte half."""
import numpy as np
import pytest
import torch

from tests.parity_util import TOL, nrel, oracle_full, run_gpu_path, say, to_dev
from workloads import NAMES, as_f64, make_inputs

pytestmark = pytest.mark.gpu

OUTS = ("O", "L", "D", "dQ", "dK", "dV", "alpha", "E", "Qt", "dOt", "Kt", "Vt")

CASES = [
    # B, H, N, d, dtype, seed, causal, form ("dq", "six" or "three")
    (1, 1, 256, 32, "f32", 120, False, "dq"),
    (1, 2, 77, 32, "f32", 121, True, "six"),
    (2, 1, 300, 32, "bf16", 122, False, "dq"),
    (1, 2, 513, 32, "bf16", 123, True, "six"),
    (1, 1, 1000, 32, "bf16", 124, False, "three"),
    (1, 1, 200, 256, "bf16", 125, False, "dq"),
    (2, 1, 97, 256, "bf16", 126, True, "dq"),
    (1, 1, 300, 256, "bf16", 127, False, "six"),
    (1, 1, 129, 256, "bf16", 128, True, "three"),
]


def case_id(c):
    return f"B{c[0]}H{c[1]}N{c[2]}d{c[3]}{c[4]}{'causal' if c[6] else ''}-{c[7]}"


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_head_dim_matches_oracle(case):
    import paper_2609_24089_amd as fb
    B, H, N, d, dt, seed, causal, form = case
    say(f"[headdim] {case_id(case)}")
    x = make_inputs(B, H, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle_full(x, scale, causal=causal)
    xd = to_dev(x)
    if form == "three":
        out = fb.bob3(*[xd[n] for n in NAMES], scale, causal=causal)
        torch.cuda.synchronize()
    else:
        out = run_gpu_path(xd, scale, use_dq=(form == "dq"), causal=causal)
    errs = {k: nrel(as_f64(out[k]), ref[k]) for k in OUTS}
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)
