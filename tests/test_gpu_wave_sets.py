"""GPU parity of the column-owned kernels (the dK, dV half of the first
backward, and Pass 2) in both of their workgroup forms: one wave set per
column block, and two wave sets that take alternate streamed tiles and add
their fp32 partial sums at the end (bob_column_opts.wave_sets).  Each form is
checked against the float64 oracle on multi-head and grouped problems, dense
and causal, with iteration counts that are odd (the second set's last
iteration has no tile) or 1 (the second set has none at all); the row-owned
outputs must not depend on the form; and the automatic choice must pick two
sets on a grid with no more workgroups than CUs and one set on a larger grid.
The wide bf16 d = 128 Pass 2 workgroups that the automatic choice runs on
large dense grids must give the one-set result bit for bit."""
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
    # B, H, Hkv, N, d, dtype, causal, seed
    (1, 2, 2, 255, 64, "bf16", False, 160),
    (1, 2, 2, 200, 128, "bf16", True, 161),
    (1, 4, 1, 161, 128, "bf16", False, 162),   # multi-query, 24 tiles per column block
    (1, 3, 1, 77, 64, "bf16", True, 163),      # 9 tiles: the second set's last iteration is empty
    (1, 1, 1, 20, 64, "bf16", False, 164),     # one tile: the second set streams nothing
    (2, 2, 1, 45, 32, "bf16", True, 165),
    (1, 2, 2, 130, 64, "f32", False, 166),
    (1, 2, 1, 100, 32, "f32", True, 167),
    (1, 2, 1, 96, 256, "bf16", False, 168),    # no room for two sets: both modes run one
]


def case_id(c):
    return f"B{c[0]}H{c[1]}kv{c[2]}N{c[3]}d{c[4]}{c[5]}{'causal' if c[6] else ''}"


@pytest.fixture
def fb():
    import paper_2609_24089_amd as m
    m.load_library()
    return m


def run(fb, xd, scale, causal, mode):
    # unsplit (Pass 2 would otherwise split these small grids over workgroups)
    out = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, columns=fb.ColumnOpts(1, mode, 0))
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_both_forms_match_oracle(fb, case):
    B, H, Hkv, N, d, dt, causal, seed = case
    say(f"[wave sets] {case_id(case)}")
    x = make_gqa_inputs(B, H, Hkv, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle.bob_gqa(*[as_f64(x[n]) for n in NAMES], scale, causal=causal)
    xd = {k: v.cuda() for k, v in x.items()}
    outs = {}
    for mode in (1, 2):
        out = run(fb, xd, scale, causal, mode)
        errs = {k: nrel(as_f64(out[k]), ref[k]) for k in OUTS}
        say(f"   mode {mode} errs", {k: f"{v:.2e}" for k, v in errs.items()})
        for k, e in errs.items():
            assert e <= TOL[dt], (mode, k, e)
        outs[mode] = out
    for k in OUTS:
        if k not in COLUMN_OUTS:
            assert torch.equal(outs[1][k], outs[2][k]), k


def column_grid(cfg_rows, B, Hkv, N):
    return B * Hkv * ((N + cfg_rows - 1) // cfg_rows)


def test_automatic_choice_follows_the_grid(fb):
    """bf16 d = 64: both column kernels own 128 key rows per workgroup.  A
    grid within the CU count must give the two-set result bit for bit, a
    larger one the one-set result."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    scale = 0.125
    small = (1, 2, 1, 300)
    Hq = 8
    n_large = 128 * (cus // (4 * Hq) + 2)
    large = (4, Hq, Hq, n_large)
    assert column_grid(128, small[0], small[2], small[3]) <= cus
    assert column_grid(128, large[0], large[2], large[3]) > cus
    for (B, H, Hkv, N), forced in ((small, 2), (large, 1)):
        say(f"[wave sets] automatic choice B{B} H{H} Hkv{Hkv} N{N} (CUs {cus}) -> mode {forced}")
        xd = {k: v.cuda() for k, v in make_gqa_inputs(B, H, Hkv, N, 64, "bf16", 170).items()}
        auto = run(fb, xd, scale, False, 0)
        ref = run(fb, xd, scale, False, forced)
        for k in OUTS:
            assert torch.equal(auto[k], ref[k]), (N, k)


def test_each_form_is_deterministic(fb):
    xd = {k: v.cuda() for k, v in make_gqa_inputs(1, 4, 1, 333, 128, "bf16", 171).items()}
    for mode in (1, 2):
        say(f"[wave sets] determinism mode {mode}")
        a = run(fb, xd, 0.1, True, mode)
        b = run(fb, xd, 0.1, True, mode)
        for k in OUTS:
            assert torch.equal(a[k], b[k]), (mode, k)


@pytest.mark.parametrize("shape", [(1, 32, 32, 2000), (1, 16, 4, 8192)], ids=["H32N2000", "H16kv4N8192"])
def test_wide_pass2_matches_one_set(fb, shape):
    """bf16 d = 128, dense: Pass 2 grids of at least one workgroup per CU in
    the wide form (128 key rows per workgroup; N = 2000 ends in a partial
    block) run wide when the wave sets are automatic and narrow (64 key rows
    per workgroup) when one set is forced; Kt and Vt must agree bit for bit
    (the same producers and Pass 1 outputs feed both)."""
    B, H, Hkv, N = shape
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert column_grid(128, B, Hkv, N) >= cus
    say(f"[wave sets] wide Pass 2 B{B} H{H} Hkv{Hkv} N{N} d128 (CUs {cus})")
    xd = {k: v.cuda() for k, v in make_gqa_inputs(B, H, Hkv, N, 128, "bf16", 172).items()}
    Q, K, V, dO, UQ, UK, UV = (xd[n] for n in NAMES)
    scale = 128 ** -0.5
    O, L = fb.attn_fwd_lse(Q, K, V, scale)
    dQ, dK, dV, D = fb.attn_bwd(Q, K, V, O, dO, L, scale)
    Qt, dOt, al, E = fb.attn_bob_pass1_rows(Q, K, V, O, dO, UQ, UK, UV, L, D, scale, dQ=dQ)
    auto = fb.attn_bob_pass2_cols(Q, K, V, dO, UQ, UK, UV, L, D, al, E, scale, columns=fb.ColumnOpts(1, 0, 0))
    one = fb.attn_bob_pass2_cols(Q, K, V, dO, UQ, UK, UV, L, D, al, E, scale, columns=fb.ColumnOpts(1, 1, 0))
    torch.cuda.synchronize()
    for a, b, name in zip(auto, one, ("Kt", "Vt")):
        assert torch.equal(a, b), name
