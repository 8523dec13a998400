"""GPU parity of Pass 2 in wave pairs (bob_pass2_pair_kernel: bf16 d = 256,
where the one-wave Pass 2 holds one wave per SIMD).  The two waves of a pair
split the head dims and hand partial score tiles and half accumulate
fragments to each other through LDS, with two workgroup-wide barriers per
tile that every wave runs.  Checked against the float64 oracle on dense and
causal, multi-head and grouped problems whose N leaves partial column blocks
and pairs with no valid key row (the automatic layout runs the pairs), and
against the one-wave form that a forced wave_sets = 1 still runs (the two
differ only in the order of fp32 sums inside the score tiles)."""
import numpy as np
import pytest
import torch

import oracle
from tests.parity_util import TOL, nrel, say
from workloads import NAMES, as_f64, make_gqa_inputs

pytestmark = pytest.mark.gpu

OUTS = ("O", "L", "D", "dQ", "dK", "dV", "alpha", "E", "Qt", "dOt", "Kt", "Vt")

CASES = [
    # B, H, Hkv, N, causal, seed
    (1, 2, 2, 200, False, 180),
    (1, 2, 2, 200, True, 181),
    (1, 4, 2, 161, True, 182),    # grouped: two query heads per key/value head
    (2, 2, 1, 77, False, 183),    # multi-query; blocks of 64 key rows, the last one partial
    (1, 1, 1, 20, True, 184),     # one tile; three of the four pairs own no valid key row
    (1, 3, 1, 300, True, 185),
]


def case_id(c):
    return f"B{c[0]}H{c[1]}kv{c[2]}N{c[3]}{'causal' if c[4] else ''}"


@pytest.fixture
def fb():
    import paper_2609_24089_amd as m
    m.load_library()
    return m


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_pairs_match_oracle_and_one_wave_form(fb, case):
    B, H, Hkv, N, causal, seed = case
    d = 256
    say(f"[pass2 pairs] {case_id(case)} d{d}")
    x = make_gqa_inputs(B, H, Hkv, N, d, "bf16", seed)
    scale = d ** -0.5
    ref = oracle.bob_gqa(*[as_f64(x[n]) for n in NAMES], scale, causal=causal)
    xd = {k: v.cuda() for k, v in x.items()}
    auto = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, columns=fb.ColumnOpts(1, 0, 0))
    one = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, columns=fb.ColumnOpts(1, 1, 0))
    torch.cuda.synchronize()
    errs = {k: nrel(as_f64(auto[k]), ref[k]) for k in OUTS}
    say("   pairs errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL["bf16"], (k, e)
    for k in ("Kt", "Vt"):
        e1 = nrel(as_f64(one[k]), ref[k])
        diff = nrel(as_f64(auto[k]), as_f64(one[k]))
        say(f"   {k}: one-wave form err {e1:.2e}, pairs vs one-wave {diff:.2e}")
        assert e1 <= TOL["bf16"] and diff <= 1e-2, (k, e1, diff)
    # the producers and Pass 1 do not depend on the Pass 2 layout
    for k in ("O", "L", "D", "dQ", "alpha", "E", "Qt", "dOt"):
        assert torch.equal(auto[k], one[k]), k
