"""GPU parity of grouped key/value heads (GQA; MQA when Hkv = 1) against the
float64 oracle `oracle.bob_gqa`: the whole path through the C ABI's grouped
entry points (chosen by the binding from the tensor shapes), every output,
dense and causal, ragged N, both dtypes and every head dim; the autograd
wrapper's Hessian-vector product with shared key/value heads; and the
benchmark's multi-query workloads at full size on sampled rows and columns."""
import numpy as np
import pytest
import torch

import oracle
from tests.parity_util import TOL, nrel, say
from workloads import NAMES, as_f64, make_gqa_inputs

pytestmark = pytest.mark.gpu

OUTS = ("O", "L", "D", "dQ", "dK", "dV", "alpha", "E", "Qt", "dOt", "Kt", "Vt")

CASES = [
    # B, H, Hkv, N, d, dtype, causal, seed
    (1, 4, 2, 255, 64, "bf16", False, 140),
    (2, 4, 1, 130, 128, "bf16", True, 141),     # multi-query
    (1, 6, 3, 300, 64, "f32", False, 142),
    (1, 8, 2, 513, 128, "bf16", False, 143),
    (1, 4, 2, 97, 256, "bf16", True, 144),
    (2, 2, 1, 200, 32, "bf16", False, 145),
    (1, 3, 1, 77, 128, "f32", True, 146),
]


def case_id(c):
    return f"B{c[0]}H{c[1]}kv{c[2]}N{c[3]}d{c[4]}{c[5]}{'causal' if c[6] else ''}"


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_grouped_heads_match_oracle(case):
    import paper_2609_24089_amd as fb
    B, H, Hkv, N, d, dt, causal, seed = case
    say(f"[gqa] {case_id(case)}")
    x = make_gqa_inputs(B, H, Hkv, N, d, dt, seed)
    scale = 1.0 / np.sqrt(d)
    ref = oracle.bob_gqa(*[as_f64(x[n]) for n in NAMES], scale, causal=causal)
    xd = {k: v.cuda() for k, v in x.items()}
    for use_dq in (True, False):
        out = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, use_dq=use_dq)
        torch.cuda.synchronize()
        errs = {k: nrel(as_f64(out[k]), ref[k]) for k in OUTS}
        say(f"   use_dq={use_dq} errs", {k: f"{v:.2e}" for k, v in errs.items()})
        for k, e in errs.items():
            assert out[k].shape == tuple(ref[k].shape), k
            assert e <= TOL[dt], (k, e)


def test_one_group_through_the_grouped_route_equals_multi_head():
    """Hkv = H through the binding is the multi-head path; and a grouped
    problem equals the multi-head path run on repeated K, V, U_K, U_V with
    Kt, Vt, dK, dV summed over each group (the same floating-point work per
    query head, so the row-owned outputs agree bit for bit)."""
    import paper_2609_24089_amd as fb
    B, H, Hkv, N, d = 1, 4, 2, 160, 64
    x = {k: v.cuda() for k, v in make_gqa_inputs(B, H, Hkv, N, d, "bf16", 147).items()}
    scale = 0.125
    out = fb.bob(*[x[n] for n in NAMES], scale)
    G = H // Hkv
    rep = {n: (x[n].repeat_interleave(G, dim=1).contiguous() if n in ("K", "V", "UK", "UV") else x[n]) for n in NAMES}
    mha = fb.bob(*[rep[n] for n in NAMES], scale)
    torch.cuda.synchronize()
    for k in ("O", "L", "D", "dQ", "alpha", "E", "Qt", "dOt"):
        assert torch.equal(out[k], mha[k]), k
    for k in ("Kt", "Vt", "dK", "dV"):
        summed = mha[k].float().reshape(B, Hkv, G, N, d).sum(dim=2)
        assert nrel(as_f64(out[k]), as_f64(summed)) <= 1e-2, k


@pytest.mark.parametrize("causal", [False, True])
def test_autograd_hvp_with_grouped_heads(causal):
    import paper_2609_24089_amd as fb
    B, H, Hkv, N, d = 1, 4, 2, 150, 64
    x = make_gqa_inputs(B, H, Hkv, N, d, "f32", 148 + int(causal))
    scale = 1.0 / np.sqrt(d)
    q, k, v = (x[n].cuda().requires_grad_(True) for n in ("Q", "K", "V"))
    u = [x[n].cuda() for n in ("UQ", "UK", "UV")]
    W = x["dO"].cuda()
    O = fb.attention(q, k, v, scale, causal)
    g = torch.autograd.grad((O * W).sum(), (q, k, v), create_graph=True)
    phi = sum((gi * ui).sum() for gi, ui in zip(g, u))
    h = torch.autograd.grad(phi, (q, k, v))
    torch.cuda.synchronize()
    ref = oracle.bob_gqa(*[as_f64(x[n]) for n in NAMES], scale, causal=causal)
    errs = {"O": nrel(as_f64(O), ref["O"])}
    for name, t in zip(("dQ", "dK", "dV"), g):
        errs[name] = nrel(as_f64(t), ref[name])
    for name, t in zip(("Qt", "Kt", "Vt"), h):
        errs[name] = nrel(as_f64(t), ref[name])
    say("   errs", {kk: f"{vv:.2e}" for kk, vv in errs.items()})
    for kk, e in errs.items():
        assert e <= TOL["f32"], (kk, e)


KV_SIDE = ("K", "V", "UK", "UV")


@pytest.mark.parametrize("name", ["mqa_bf16_b1h16kv1_n16384_d128", "causal_mqa_bf16_b1h16kv1_n16384_d128"])
def test_multi_query_at_full_size(name):
    """The multi-query workloads of the benchmark (B1, 16 query heads sharing
    one key/value head, N = 16384, d = 128), run as the benchmark runs them
    (its column kernels then split each column block over several
    workgroups, with a workspace and a reduction).  Row-owned outputs
    on 32 sampled query rows of every head against the oracle; column-owned
    outputs (Kt, Vt, dK, dV) on 64 sampled key rows, against the oracle's
    column slices summed over the 16 query heads, given the GPU's row scalars
    (which the sampled-row check covers); the identities I1-I3, I5, I6 on the
    full outputs."""
    from tests.parity_util import check_identities
    from workloads import WORKLOADS, workload_inputs
    w = WORKLOADS[name]
    G = w.H // w.kv_heads
    say(f"[gqa] {w.name}: GPU path")
    x = workload_inputs(w)
    xd = {k: v.cuda() for k, v in x.items()}
    import paper_2609_24089_amd as fb
    out = fb.bob(*[xd[n] for n in NAMES], w.scale, causal=w.causal)
    torch.cuda.synchronize()
    head = lambda h: [as_f64(x[n][0, h // G if n in KV_SIDE else h]) for n in NAMES]
    rng = np.random.default_rng(3001)
    row_keys = ("Qt", "dOt", "alpha", "E", "O", "L", "D", "dQ")
    got, want = {k: [] for k in row_keys}, {k: [] for k in row_keys}
    for h in range(w.H):
        rows = np.unique(np.concatenate([[0], rng.choice(w.N, size=32, replace=False)]))
        ref = oracle.bob_rows(*head(h), w.scale, rows, causal=w.causal)
        idx = torch.as_tensor(rows, device=out["Qt"].device)
        for k in row_keys:
            got[k].append(as_f64(out[k][0, h].index_select(0, idx)))
            want[k].append(ref[k])
    errs = {k: nrel(np.concatenate(got[k]), np.concatenate(want[k])) for k in row_keys}
    say("   sampled-row errs", {k: f"{v:.2e}" for k, v in errs.items()})
    cols = np.sort(np.random.default_rng(3002).choice(w.N, size=64, replace=False))
    col_keys = ("Kt", "Vt", "dK", "dV")
    acc = {k: 0.0 for k in col_keys}
    for h in range(w.H):
        rs = {k: as_f64(out[k][0, h]) for k in ("alpha", "E", "L", "D")}
        ref = oracle.bob_cols(*head(h), w.scale, cols, rs["alpha"], rs["E"], rs["L"], rs["D"], causal=w.causal)
        for k in col_keys:
            acc[k] = acc[k] + ref[k]
    idx = torch.as_tensor(cols, device=out["Kt"].device)
    for k in col_keys:
        errs[k] = nrel(as_f64(out[k][0, 0].index_select(0, idx)), acc[k])
    say("   errs with sampled columns", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL["bf16"], (k, e)
    check_identities(xd, out)
