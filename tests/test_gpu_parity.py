"""GPU parity: the HIP path (through the C ABI) against the float64 oracle,
element by element, at sizes the oracle finishes in seconds.  The shapes span
several workgroup tiles and ragged tails (N not a multiple of the 32-row
streamed tile or of the 64/128-row stationary block), both head dims, both
dtypes and B*H > 1.  Bars: normwise relative error <= 1e-4 (fp32) and
<= 2e-2 (bf16 inputs, fp32 accumulation)."""
import numpy as np
import pytest
import torch

from tests.parity_util import TOL, lib, nrel, oracle_full, run_gpu_path, say, to_dev
from workloads import NAMES, WORKLOADS, as_f64, make_inputs, workload_inputs

pytestmark = pytest.mark.gpu

OUTS = ("O", "L", "D", "dQ", "dK", "dV", "alpha", "E", "Qt", "dOt", "Kt", "Vt")

CASES = [
    # B, H, N, d, dtype, seed
    (1, 1, 256, 64, "f32", 0),     # the tiny fp32 workload
    (1, 1, 17, 64, "f32", 11),
    (1, 2, 255, 128, "f32", 12),
    (2, 1, 300, 128, "f32", 13),
    (1, 1, 33, 64, "bf16", 14),
    (2, 1, 257, 64, "bf16", 15),
    (1, 1, 1000, 128, "bf16", 16),
    (2, 3, 100, 64, "bf16", 17),
    (1, 2, 513, 128, "bf16", 18),
]


def case_id(c):
    return f"B{c[0]}H{c[1]}N{c[2]}d{c[3]}{c[4]}s{c[5]}"


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_full_path_matches_oracle(case):
    B, H, N, d, dt, seed = case
    say(f"[parity] full path {case_id(case)}")
    x = make_inputs(B, H, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle_full(x, scale)
    out = run_gpu_path(to_dev(x), scale)
    errs = {k: nrel(as_f64(out[k]), ref[k]) for k in OUTS}
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)


@pytest.mark.parametrize("case", [(1, 1, 255, 64, "f32", 51), (1, 2, 300, 128, "f32", 52),
                                  (2, 1, 257, 64, "bf16", 53), (1, 2, 513, 128, "bf16", 54)], ids=case_id)
def test_six_accumulator_form_matches_oracle(case):
    """Pass 1 without dQ: the six row accumulators of Prop. 3.1 (R accumulated)."""
    B, H, N, d, dt, seed = case
    say(f"[parity] six-accumulator Pass 1 {case_id(case)}")
    x = make_inputs(B, H, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle_full(x, scale)
    out = run_gpu_path(to_dev(x), scale, use_dq=False)
    errs = {k: nrel(as_f64(out[k]), ref[k]) for k in ("Qt", "dOt", "alpha", "E", "Kt", "Vt")}
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)


@pytest.mark.parametrize("case", [(1, 1, 40, 64, "f32", 21), (1, 1, 200, 128, "bf16", 22),
                                  (2, 2, 130, 64, "bf16", 23)], ids=case_id)
def test_bob_passes_with_oracle_row_state(case):
    """Pass 1 and Pass 2 alone, fed the oracle's O, L, D (O cast to the input dtype)."""
    B, H, N, d, dt, seed = case
    say(f"[parity] passes with oracle state {case_id(case)}")
    fb = lib()
    x = make_inputs(B, H, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle_full(x, scale)
    xd = to_dev(x)
    tdt = xd["Q"].dtype
    O = torch.from_numpy(ref["O"]).to(tdt).cuda()
    L = torch.from_numpy(ref["L"]).float().cuda()
    D = torch.from_numpy(ref["D"]).float().cuda()
    Qt, dOt, alpha, E = fb.attn_bob_pass1_rows(xd["Q"], xd["K"], xd["V"], O, xd["dO"], xd["UQ"],
                                               xd["UK"], xd["UV"], L, D, scale)
    Kt, Vt = fb.attn_bob_pass2_cols(xd["Q"], xd["K"], xd["V"], xd["dO"], xd["UQ"], xd["UK"],
                                    xd["UV"], L, D, alpha, E, scale)
    torch.cuda.synchronize()
    got = dict(Qt=Qt, dOt=dOt, alpha=alpha, E=E, Kt=Kt, Vt=Vt)
    errs = {k: nrel(as_f64(v), ref[k]) for k, v in got.items()}
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_single_token(dt):
    """N = 1: P = [1], so Qt = Kt = Vt = 0 and dOt = U_V exactly (in exact arithmetic)."""
    say(f"[parity] N=1 {dt}")
    x = make_inputs(1, 2, 1, 64, dt, 31)
    out = run_gpu_path(to_dev(x), 0.125)
    assert nrel(as_f64(out["dOt"]), as_f64(x["UV"])) <= TOL[dt]
    lim = 1e-4 if dt == "f32" else 5e-2
    for k in ("Qt", "Kt", "Vt"):
        assert np.abs(as_f64(out[k])).max() <= lim, k
    np.testing.assert_allclose(as_f64(out["L"]), (as_f64(x["Q"]) * as_f64(x["K"])).sum(-1) * 0.125,
                               rtol=1e-5, atol=1e-5)


def test_small_bf16_workload_full_oracle():
    """The B=2, H=8, N=4096, d=64 bf16 workload (seed 1), every output element."""
    w = WORKLOADS["bf16_b2h8_n4096_d64"]
    say(f"[parity] workload {w.name}")
    x = workload_inputs(w)
    out = run_gpu_path(to_dev(x), w.scale)
    ref = oracle_full(x, w.scale)
    errs = {k: nrel(as_f64(out[k]), ref[k]) for k in OUTS}
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL["bf16"], (k, e)


def test_deterministic_bitwise():
    """No atomics anywhere: two runs give bit-identical outputs."""
    say("[parity] determinism")
    x = to_dev(make_inputs(1, 4, 777, 128, "bf16", 41))
    a = run_gpu_path(x, 0.1)
    b = run_gpu_path(x, 0.1)
    for k in OUTS:
        assert torch.equal(a[k], b[k]), k


GRID_CASES = [
    # B, H, N, d, dtype, seed, causal: many heads, workgroup counts that are
    # and are not multiples of the 8 XCDs (the block remap has both paths)
    (5, 13, 41, 64, "bf16", 140, False),
    (8, 8, 200, 128, "bf16", 141, False),
    (3, 7, 100, 128, "bf16", 142, True),
    (16, 4, 64, 64, "f32", 143, True),
]


@pytest.mark.parametrize("case", GRID_CASES, ids=lambda c: f"B{c[0]}H{c[1]}N{c[2]}d{c[3]}{c[4]}{'c' if c[6] else ''}")
def test_many_heads_grid_mapping(case):
    B, H, N, d, dt, seed, causal = case
    say(f"[grid] B{B} H{H} N{N} d{d} {dt} causal={causal}")
    x = make_inputs(B, H, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle_full(x, scale, causal=causal)
    out = run_gpu_path(to_dev(x), scale, causal=causal)
    errs = {k: nrel(as_f64(out[k]), ref[k]) for k in ("O", "L", "dQ", "dK", "dV", "alpha", "E", "Qt", "dOt", "Kt", "Vt")}
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)
