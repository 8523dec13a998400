"""GPU parity of the column kernels (the first backward's dK, dV and Pass
2's Kt, Vt) with each key/value column block split over several workgroups
(attn_bwd_gqa_ws, attn_bob_pass2_cols_gqa_ws; forced with
bob_column_opts.parts):
every split is checked against the float64 oracle on multi-head and grouped
problems, dense and causal, including splits into more parts than a block
has (query head, query tile) iterations, so that some parts stream nothing
and store zeros; the row-owned outputs must not depend on the split, and dK,
dV, Kt, Vt must agree with the unsplit kernels to the rounding of the fp32
sums."""
import ctypes

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
    (1, 2, 2, 255, 64, "bf16", True, 170),
    (1, 4, 1, 161, 128, "bf16", True, 171),    # multi-query, 6 tiles per head
    (1, 4, 1, 161, 128, "bf16", False, 172),
    (2, 6, 2, 200, 32, "bf16", True, 173),
    (1, 2, 1, 20, 64, "bf16", True, 174),      # 1 tile per head, 2 iterations: parts 2.. stream nothing
    (1, 2, 2, 130, 64, "f32", True, 175),
    (1, 2, 1, 100, 128, "f32", False, 176),
    (1, 2, 1, 96, 256, "bf16", True, 177),     # one-wave-per-SIMD shape
]


def case_id(c):
    return f"B{c[0]}H{c[1]}kv{c[2]}N{c[3]}d{c[4]}{c[5]}{'causal' if c[6] else ''}"


@pytest.fixture
def fb():
    import paper_2609_24089_amd as m
    m.load_library()
    return m


def ws_bytes(fb, pass2, code, B, H, Hkv, N, d, causal, columns=None):
    lib = fb.load_library()
    q = lib.bob_pass2_workspace_bytes if pass2 else lib.bob_bwd_workspace_bytes
    return q(code, B, H, Hkv, N, d, int(causal), None if columns is None else ctypes.byref(columns))


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_split_matches_oracle_and_unsplit(fb, case):
    B, H, Hkv, N, d, dt, causal, seed = case
    say(f"[column split] {case_id(case)}")
    x = make_gqa_inputs(B, H, Hkv, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle.bob_gqa(*[as_f64(x[n]) for n in NAMES], scale, causal=causal)
    xd = {k: v.cuda() for k, v in x.items()}
    code = fb.BOB_BF16 if dt == "bf16" else fb.BOB_F32
    one = fb.ColumnOpts(1, 1, 0)
    assert ws_bytes(fb, True, code, B, H, Hkv, N, d, causal, one) == 0
    assert ws_bytes(fb, False, code, B, H, Hkv, N, d, causal, one) == 0
    base = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, columns=one)
    torch.cuda.synchronize()
    for parts in (2, 3, 8):
        cols = fb.ColumnOpts(parts, 0, 0)
        want = parts * 2 * B * Hkv * N * d * 4
        assert ws_bytes(fb, True, code, B, H, Hkv, N, d, causal, cols) == want
        assert ws_bytes(fb, False, code, B, H, Hkv, N, d, causal, cols) == want
        out = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, columns=cols)
        torch.cuda.synchronize()
        errs = {k: nrel(as_f64(out[k]), ref[k]) for k in OUTS}
        say(f"   parts {parts} errs", {k: f"{v:.2e}" for k, v in errs.items()})
        for k, e in errs.items():
            assert e <= TOL[dt], (parts, k, e)
        for k in OUTS:
            if k not in COLUMN_OUTS:
                assert torch.equal(out[k], base[k]), (parts, k)
        for k in COLUMN_OUTS:
            diff = nrel(as_f64(out[k]), as_f64(base[k]))
            assert diff <= (1e-2 if dt == "bf16" else 1e-5), (parts, k, diff)


def test_split_on_a_side_stream(fb):
    """The binding's workspace is kept from reuse until the kernels on the
    caller's stream are done; results on a non-current stream equal those on
    the current one."""
    x = make_gqa_inputs(1, 4, 1, 300, 128, "bf16", 178)
    xd = {k: v.cuda() for k, v in x.items()}
    Q, K, V, dO, UQ, UK, UV = (xd[n] for n in NAMES)
    scale = 128 ** -0.5
    O, L = fb.attn_fwd_lse(Q, K, V, scale, True)
    dQ, dK, dV, D = fb.attn_bwd(Q, K, V, O, dO, L, scale, True)
    Qt, dOt, al, E = fb.attn_bob_pass1_rows(Q, K, V, O, dO, UQ, UK, UV, L, D, scale, True, dQ=dQ)
    cols = fb.ColumnOpts(4, 0, 0)
    ref = fb.attn_bob_pass2_cols(Q, K, V, dO, UQ, UK, UV, L, D, al, E, scale, True, columns=cols)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    outs = []
    for _ in range(3):
        outs.append(fb.attn_bob_pass2_cols(Q, K, V, dO, UQ, UK, UV, L, D, al, E, scale, True, stream=side,
                                           columns=cols))
    side.synchronize()
    for kt, vt in outs:
        assert torch.equal(kt, ref[0]) and torch.equal(vt, ref[1])


def test_automatic_choice(fb):
    """Automatic parts split a causal grid up to about 8 jobs per CU (at most 8
    parts); Pass 2 splits a dense grid only when it has fewer workgroups than
    CUs, the first backward to about 8 jobs per CU as well; blocks of fewer
    than 1024 streamed iterations and the multi-head workloads stay
    unsplit; the automatic result equals the forced one bit for bit."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    N, d = 16384, 128
    grid = lambda Hkv: Hkv * (N // 64)          # bf16 d = 128 Pass 2: 64 key rows per workgroup
    expect = lambda g, causal: (min(8, -(-8 * cus // g)) if causal else
                                (min(8, -(-2 * cus // g)) if g <= cus else 1))
    for Hkv, causal in ((1, 1), (1, 0), (4, 1), (4, 0), (16, 1), (16, 0)):
        parts = expect(grid(Hkv), causal)
        parts = parts if parts >= 2 else 1
        want = 0 if parts == 1 else parts * 2 * Hkv * N * d * 4
        got = ws_bytes(fb, True, fb.BOB_BF16, 1, 16, Hkv, N, d, causal)
        say(f"[column split] auto Hkv={Hkv} causal={causal} CUs {cus}: {got} bytes (parts {parts})")
        assert got == want, (Hkv, causal, got, want)
        # the first backward's column kernel owns 128 key rows per workgroup
        # here (32 per wave), and is split to about 8 jobs per CU under
        # either mask
        pb = min(8, -(-8 * cus // (Hkv * (N // 128))))
        want_b = 0 if pb < 2 else pb * 2 * Hkv * N * d * 4
        assert ws_bytes(fb, False, fb.BOB_BF16, 1, 16, Hkv, N, d, causal) == want_b, (Hkv, causal)
    # short blocks (fewer than 1024 streamed iterations) are never split
    for Hkv, n in ((12, 4096), (12, 2048), (1, 500)):
        for causal in (0, 1):
            assert ws_bytes(fb, True, fb.BOB_BF16, 4, 12 if Hkv == 12 else 4, Hkv, n, 64, causal) == 0
            assert ws_bytes(fb, False, fb.BOB_BF16, 4, 12 if Hkv == 12 else 4, Hkv, n, 64, causal) == 0
    # a causal multi-query problem with 16 x 64 = 1024 iterations per block:
    # automatic equals the forced part count
    B, H, Hkv, n = 1, 16, 1, 2048
    g = -(-n // 64)
    parts = min(8, -(-8 * cus // g))
    xd = {k: v.cuda() for k, v in make_gqa_inputs(B, H, Hkv, n, 128, "bf16", 179).items()}
    auto = fb.bob(*[xd[k] for k in NAMES], 0.1, causal=True)
    forced = fb.bob(*[xd[k] for k in NAMES], 0.1, causal=True, columns=fb.ColumnOpts(parts, 0, 0))
    torch.cuda.synchronize()
    for k in OUTS:
        assert torch.equal(auto[k], forced[k]), k


def test_automatic_workspace_is_bounded(fb):
    """The automatic split only triggers on grids smaller than about 8 jobs
    per CU, so its workspace (parts x 2 x B*Hkv*N*d fp32) stays bounded as N
    grows: at most 8 x CUs x (key rows per workgroup) x 2 x d x 4 bytes for
    the parts plus one block's rounding, whatever N (multi-query, causal and
    dense, d = 64 and 128, N = 2^10 ... 2^22)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    worst = 0
    for d in (64, 128):
        for causal in (False, True):
            for logn in range(10, 23):
                for kernel in (fb.BOB_COLUMNS_BWD, fb.BOB_COLUMNS_PASS2):
                    lay, nbytes = fb.column_layout(kernel, torch.bfloat16, 1, 16, 1, 1 << logn, d, causal)
                    worst = max(worst, nbytes)
                    bound = 2 * 8 * cus * 128 * 2 * d * 4
                    assert nbytes <= bound, (d, causal, logn, kernel, lay, nbytes)
    say(f"[column split] largest automatic workspace over the sweep: {worst / 2**20:.0f} MiB on {cus} CUs")


def test_long_causal_multi_query_split_and_footprint(fb):
    """Causal multi-query attention at N = 65536 (B1, 16 query heads sharing
    one key/value head, d = 64), where both column kernels split each block
    over several workgroups: row-owned outputs on 16 uniformly sampled query
    rows of every head (and row 0, whose Qt is exactly zero, against the
    bound of its one bf16 rounding) and column-owned outputs on 32 sampled key rows (summed over the
    query heads, given the GPU's row scalars, which the row check covers)
    against the oracle, and the identities I1-I3, I5, I6.  Footprint: the first
    backward adds exactly its workspace to the device memory in use, Pass 1
    nothing beyond its outputs, and Pass 2 exactly its workspace."""
    from tests.parity_util import check_identities
    B, H, Hkv, N, d, causal = 1, 16, 1, 65536, 64, True
    G = H // Hkv
    scale = d ** -0.5
    x = make_gqa_inputs(B, H, Hkv, N, d, "bf16", 193)
    xd = {k: v.cuda() for k, v in x.items()}
    Q, K, V, dO, UQ, UK, UV = (xd[n] for n in NAMES)
    lays = {k: fb.column_layout(k, torch.bfloat16, B, H, Hkv, N, d, causal) for k in (fb.BOB_COLUMNS_BWD,
                                                                                     fb.BOB_COLUMNS_PASS2)}
    say(f"[column split] long causal MQA N={N}: layouts {lays}")
    assert all(lay.parts >= 2 for lay, _ in lays.values())
    O, L = fb.attn_fwd_lse(Q, K, V, scale, causal)
    outs_b = (torch.empty_like(Q), torch.empty_like(K), torch.empty_like(K), torch.empty_like(L))
    outs_1 = (torch.empty_like(Q), torch.empty_like(Q), torch.empty_like(L), torch.empty_like(L))
    outs_2 = (torch.empty_like(K), torch.empty_like(K))

    def extra(fn):
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        fn()
        torch.cuda.synchronize()
        return torch.cuda.max_memory_allocated() - before

    eb = extra(lambda: fb.attn_bwd(Q, K, V, O, dO, L, scale, causal, out=outs_b))
    dQ, dK, dV, D = outs_b
    e1 = extra(lambda: fb.attn_bob_pass1_rows(Q, K, V, O, dO, UQ, UK, UV, L, D, scale, causal, dQ=dQ, out=outs_1))
    Qt, dOt, al, E = outs_1
    e2 = extra(lambda: fb.attn_bob_pass2_cols(Q, K, V, dO, UQ, UK, UV, L, D, al, E, scale, causal, out=outs_2))
    say(f"   extra device memory: bwd {eb >> 20} MiB, Pass 1 {e1}, Pass 2 {e2 >> 20} MiB; alpha + E "
        f"{(al.nbytes + E.nbytes) >> 20} MiB")
    assert eb == lays[fb.BOB_COLUMNS_BWD][1] and e1 == 0 and e2 == lays[fb.BOB_COLUMNS_PASS2][1]
    assert al.nbytes + E.nbytes == 2 * 4 * B * H * N
    out = dict(O=O, L=L, D=D, dQ=dQ, dK=dK, dV=dV, Qt=Qt, dOt=dOt, alpha=al, E=E, Kt=outs_2[0], Vt=outs_2[1])
    head = lambda h: [as_f64(x[n][0, h // G if n in ("K", "V", "UK", "UV") else h]) for n in NAMES]
    rng = np.random.default_rng(3101)
    row_keys = ("Qt", "dOt", "alpha", "E", "O", "L", "D", "dQ")
    got, want = {k: [] for k in row_keys}, {k: [] for k in row_keys}
    for h in range(H):
        rows = np.unique(rng.choice(N, size=16, replace=False))
        ref = oracle.bob_rows(*head(h), scale, rows, causal=causal)
        idx = torch.as_tensor(rows, device=Q.device)
        for k in row_keys:
            got[k].append(as_f64(out[k][0, h].index_select(0, idx)))
            want[k].append(ref[k])
        # Row 0 sees key 0 only, where Qt is exactly 0: what remains is the
        # rounding of the one bf16 operand P Pt0 = C_00 (times tau k_0) that
        # the affine form's Omega - E0 B cancels against its fp32 row sum, at
        # most 2^-8 |C_00| |k_0| tau, with |C_00| <= |dO_0| |U_V,0|.
        q, k0, v, do, uq, uk, uv = head(h)
        ref0 = oracle.bob_rows(q, k0, v, do, uq, uk, uv, scale, np.array([0]), causal=causal)
        bound = 2.0 ** -8 * scale * np.linalg.norm(do[0]) * np.linalg.norm(uv[0]) * np.linalg.norm(k0[0])
        assert np.abs(ref0["Qt"]).max() == 0.0
        assert np.linalg.norm(as_f64(out["Qt"][0, h, 0]) - ref0["Qt"][0]) <= bound, h
    errs = {k: nrel(np.concatenate(got[k]), np.concatenate(want[k])) for k in row_keys}
    cols = np.sort(np.random.default_rng(3102).choice(N, size=32, replace=False))
    acc = {k: 0.0 for k in COLUMN_OUTS}
    for h in range(H):
        rs = {k: as_f64(out[k][0, h]) for k in ("alpha", "E", "L", "D")}
        ref = oracle.bob_cols(*head(h), scale, cols, rs["alpha"], rs["E"], rs["L"], rs["D"], causal=causal)
        for k in COLUMN_OUTS:
            acc[k] = acc[k] + ref[k]
    idx = torch.as_tensor(cols, device=Q.device)
    for k in COLUMN_OUTS:
        errs[k] = nrel(as_f64(out[k][0, 0].index_select(0, idx)), acc[k])
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL["bf16"], (k, e)
    check_identities(xd, out)
