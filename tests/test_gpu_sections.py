"""GPU parity of the column kernels' sectioned accumulation (the first
backward's dK, dV and Pass 2's Kt, Vt; bob_column_opts.flush_tiles): the
MFMA accumulator chain restarts every `flush_tiles` streamed tiles and is
added into fp32 sums by round-to-nearest VALU adds.  Forced to sections of
one to a few tiles at small N, every layout it combines with (multi-head and
grouped heads, dense and causal, unsplit with one or two wave sets, split
into parts, d = 32, 64, 128) is checked against the float64 oracle, and
against the one-section result to the rounding of the fp32 sums; the
row-owned outputs must not change.  (dtype, d) pairs without a sectioned
form refuse a request for sections.  The automatic choice at long N is
covered by tests/test_gpu_peak_n.py and, without a GPU, by
tests/test_abi_cpu.py."""
import numpy as np
import pytest
import torch

import oracle
from tests.parity_util import TOL, nrel, say
from workloads import NAMES, as_f64, make_gqa_inputs

pytestmark = pytest.mark.gpu

OUTS = ("O", "L", "D", "dQ", "dK", "dV", "alpha", "E", "Qt", "dOt", "Kt", "Vt")
COLUMN_OUTS = ("dK", "dV", "Kt", "Vt")

CASES = [
    # B, H, Hkv, N, d, causal, seed, (parts, wave_sets, flush_tiles)
    (1, 2, 2, 255, 64, False, 180, (1, 1, 1)),
    (1, 2, 2, 255, 64, True, 181, (1, 1, 3)),
    (1, 4, 1, 161, 128, False, 182, (1, 1, 2)),     # grouped: 4 x 6 streamed tiles
    (1, 4, 1, 161, 128, True, 183, (1, 2, 2)),      # two wave sets
    (2, 6, 2, 200, 32, True, 184, (1, 1, 1)),
    (2, 6, 2, 200, 32, False, 185, (3, 1, 1)),      # split into parts
    (1, 3, 1, 77, 64, True, 186, (2, 1, 4)),        # more sections than some parts stream
    (1, 2, 2, 300, 128, True, 187, (1, 1, 5)),
]


def case_id(c):
    return f"B{c[0]}H{c[1]}kv{c[2]}N{c[3]}d{c[4]}{'causal' if c[5] else ''}-opts{c[7]}"


@pytest.fixture
def fb():
    import paper_2609_24089_amd as m
    m.load_library()
    return m


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_sections_match_oracle(fb, case):
    B, H, Hkv, N, d, causal, seed, (parts, sets, flush) = case
    say(f"[sections] {case_id(case)}")
    x = make_gqa_inputs(B, H, Hkv, N, d, "bf16", seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle.bob_gqa(*[as_f64(x[n]) for n in NAMES], scale, causal=causal)
    xd = {k: v.cuda() for k, v in x.items()}
    one = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, columns=fb.ColumnOpts(parts, sets, -1))
    sec = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, columns=fb.ColumnOpts(parts, sets, flush))
    torch.cuda.synchronize()
    for kernel in (fb.BOB_COLUMNS_BWD, fb.BOB_COLUMNS_PASS2):
        got, _ = fb.column_layout(kernel, torch.bfloat16, B, H, Hkv, N, d, causal,
                                  fb.ColumnOpts(parts, sets, flush))
        assert got.flush_tiles == flush, (kernel, got)
    errs = {k: nrel(as_f64(sec[k]), ref[k]) for k in OUTS}
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL["bf16"], (k, e)
    for k in OUTS:
        if k not in COLUMN_OUTS:
            assert torch.equal(sec[k], one[k]), k
    for k in COLUMN_OUTS:
        diff = nrel(as_f64(sec[k]), as_f64(one[k]))
        assert diff <= 1e-2, (k, diff)


@pytest.mark.parametrize("dt,d", [("bf16", 256), ("f32", 64)])
def test_sections_refused_where_not_built(fb, dt, d):
    x = make_gqa_inputs(1, 2, 2, 64, d, dt, 188)
    xd = {k: v.cuda() for k, v in x.items()}
    with pytest.raises(RuntimeError, match="BOB_EUNSUPPORTED"):
        fb.bob(*[xd[n] for n in NAMES], 1.0 / np.sqrt(d), columns=fb.ColumnOpts(1, 1, 4))
    torch.cuda.synchronize()
