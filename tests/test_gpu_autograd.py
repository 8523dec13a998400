"""GPU checks of the autograd wrapper (`paper_2609_24089_amd.attention`):
first and second reverse-mode derivatives routed through the HIP kernels,
compared with the float64 oracle.

* loss <O, W>: dO = W is constant, so the Hessian-vector product in
  (Q, K, V) along (U_Q, U_K, U_V) is exactly BoB's (Qt, Kt, Vt) (Sec. 3.1).
* loss <O, W> + |O|^2 / 2: dO = W + O depends on Q, K, V, so the product
  adds the first backward of attention taken with upstream dOt (BoB's dO
  cotangent) -- the term the wrapper routes into the graph of dO.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.parity_util import TOL, nrel, say
from workloads import as_f64, make_inputs

pytestmark = pytest.mark.gpu

CASES = [
    # B, H, N, d, dtype, seed, causal
    (1, 2, 200, 64, "f32", 80, False),
    (2, 1, 97, 128, "f32", 81, True),
    (1, 2, 300, 64, "bf16", 82, False),
    (1, 1, 257, 128, "bf16", 83, True),
]


def case_id(c):
    return f"B{c[0]}H{c[1]}N{c[2]}d{c[3]}{c[4]}{'causal' if c[6] else ''}"


def hvp_gpu(x, W, scale, causal, curvature):
    import paper_2609_24089_amd as fb
    q, k, v = (x[n].cuda().requires_grad_(True) for n in ("Q", "K", "V"))
    u = [x[n].cuda() for n in ("UQ", "UK", "UV")]
    Wd = W.cuda()
    O = fb.attention(q, k, v, scale, causal)
    loss = (O.float() * Wd.float()).sum()
    if curvature:
        loss = loss + 0.5 * (O.float() ** 2).sum()
    g = torch.autograd.grad(loss, (q, k, v), create_graph=True)
    phi = sum((gi.float() * ui.float()).sum() for gi, ui in zip(g, u))
    h = torch.autograd.grad(phi, (q, k, v))
    torch.cuda.synchronize()
    return O, g, h


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_hvp_of_linear_loss_is_bob(case):
    B, H, N, d, dt, seed, causal = case
    say(f"[autograd] linear loss {case_id(case)}")
    x = make_inputs(B, H, N, d, dt, seed)
    W = x["dO"]
    scale = 1.0 / np.sqrt(d)
    O, g, h = hvp_gpu(x, W, scale, causal, curvature=False)
    args = [as_f64(x[n]) for n in ("Q", "K", "V", "dO", "UQ", "UK", "UV")]
    ref = oracle.bob(*args, scale, causal=causal)
    errs = {"O": nrel(as_f64(O), ref["O"])}
    for name, t in zip(("dQ", "dK", "dV"), g):
        errs[name] = nrel(as_f64(t), ref[name])
    for name, t in zip(("Qt", "Kt", "Vt"), h):
        errs[name] = nrel(as_f64(t), ref[name])
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)


@pytest.mark.parametrize("case", CASES, ids=case_id)
def test_hvp_with_curvature_in_the_loss(case):
    B, H, N, d, dt, seed, causal = case
    say(f"[autograd] loss with curvature {case_id(case)}")
    x = make_inputs(B, H, N, d, dt, seed + 100)
    W = x["dO"]
    scale = 1.0 / np.sqrt(d)
    O, g, h = hvp_gpu(x, W, scale, causal, curvature=True)
    q, k, v, w, uq, uk, uv = [as_f64(x[n]) for n in ("Q", "K", "V", "dO", "UQ", "UK", "UV")]
    Oref = oracle.forward(q, k, v, scale, causal=causal)["O"]
    dO = w + Oref                                   # gradient of the loss in O
    ref = oracle.bob(q, k, v, dO, uq, uk, uv, scale, causal=causal)
    extra = oracle.first_backward(q, k, v, ref["dOt"], scale, causal=causal)
    want = {"dQ": ref["dQ"], "dK": ref["dK"], "dV": ref["dV"],
            "Qt": ref["Qt"] + extra["dQ"], "Kt": ref["Kt"] + extra["dK"], "Vt": ref["Vt"] + extra["dV"]}
    got = dict(zip(("dQ", "dK", "dV"), g)) | dict(zip(("Qt", "Kt", "Vt"), h))
    errs = {name: nrel(as_f64(got[name]), want[name]) for name in want}
    say("   errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL[dt], (k, e)


def test_partial_requires_grad():
    """Only K requires grad: the second derivative reaches K alone."""
    import paper_2609_24089_amd as fb
    x = make_inputs(1, 1, 130, 64, "f32", 90)
    scale = 0.125
    q, v = x["Q"].cuda(), x["V"].cuda()
    k = x["K"].cuda().requires_grad_(True)
    O = fb.attention(q, k, v, scale)
    (gk,) = torch.autograd.grad((O * x["dO"].cuda()).sum(), (k,), create_graph=True)
    (hk,) = torch.autograd.grad((gk * x["UK"].cuda()).sum(), (k,))
    zero = np.zeros_like(as_f64(x["Q"]))
    args = [as_f64(x[n]) for n in ("Q", "K", "V", "dO")]
    ref = oracle.bob(*args, zero, as_f64(x["UK"]), zero, scale)
    e = nrel(as_f64(hk), ref["Kt"])
    say("   Kt err", f"{e:.2e}")
    assert e <= TOL["f32"]
