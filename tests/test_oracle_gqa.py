"""Pins for the grouped-query (GQA / MQA) oracle, `oracle.bob_gqa`.

* torch's own double backward in float64 through a GQA forward that repeats
  K and V per query head inside the graph (so autograd, not the oracle, sums
  the key/value-side gradients over each group);
* G = 1 is multi-head attention;
* the global identities I1-I3, which follow from linearity in dO, linearity
  of dQ, dK in V, and the invariance of S under Q -> cQ, K -> K / c, and so
  hold with shared key/value heads too;
* planted grouping mistakes break the torch pin."""
import numpy as np
import pytest
import torch

import oracle
from oracle import bob_oracle as bo

TOL = 1e-11


def inputs(B, Hq, Hkv, N, d, seed):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, Hq, N, d))
    k = rng.standard_normal((B, Hkv, N, d))
    v = rng.standard_normal((B, Hkv, N, d))
    do = rng.standard_normal((B, Hq, N, d))
    uq = rng.standard_normal((B, Hq, N, d))
    uk = rng.standard_normal((B, Hkv, N, d))
    uv = rng.standard_normal((B, Hkv, N, d))
    return q, k, v, do, uq, uk, uv


def torch_gqa_bob(q, k, v, do, uq, uk, uv, tau, causal):
    G = q.shape[1] // k.shape[1]
    Q, K, V, dO = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (q, k, v, do))
    UQ, UK, UV = (torch.tensor(a, dtype=torch.float64) for a in (uq, uk, uv))
    Kx, Vx = K.repeat_interleave(G, dim=1), V.repeat_interleave(G, dim=1)
    S = tau * (Q @ Kx.transpose(-1, -2))
    if causal:
        n = S.shape[-1]
        S = S.masked_fill(torch.ones(n, n, dtype=torch.bool).triu(1), float("-inf"))
    O = torch.softmax(S, dim=-1) @ Vx
    dQ, dK, dV = torch.autograd.grad(O, (Q, K, V), grad_outputs=dO, create_graph=True)
    phi = (dQ * UQ).sum() + (dK * UK).sum() + (dV * UV).sum()
    Qt, Kt, Vt, dOt = torch.autograd.grad(phi, (Q, K, V, dO))
    return dict(O=O.detach().numpy(), dQ=dQ.detach().numpy(), dK=dK.detach().numpy(), dV=dV.detach().numpy(),
                Qt=Qt.numpy(), Kt=Kt.numpy(), Vt=Vt.numpy(), dOt=dOt.numpy(), phi=float(phi.detach()))


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


@pytest.mark.parametrize("B,Hq,Hkv,N,d,causal,seed", [
    (1, 4, 2, 23, 8, False, 1), (2, 4, 1, 17, 4, True, 2), (1, 6, 3, 9, 5, True, 3), (1, 3, 3, 11, 4, False, 4)])
def test_gqa_oracle_matches_torch_double_backward(B, Hq, Hkv, N, d, causal, seed):
    x = inputs(B, Hq, Hkv, N, d, seed)
    tau = 1.0 / np.sqrt(d)
    ref = oracle.bob_gqa(*x, tau, causal=causal)
    tb = torch_gqa_bob(*x, tau, causal)
    for key in ("O", "dQ", "dK", "dV", "Qt", "Kt", "Vt", "dOt"):
        assert ref[key].shape == tb[key].shape, key
        assert rel(ref[key], tb[key]) <= TOL, (key, rel(ref[key], tb[key]))


def test_one_group_is_multi_head():
    x = inputs(2, 3, 3, 13, 4, 5)
    a = oracle.bob_gqa(*x, 0.4, causal=True)
    b = oracle.bob(*x, 0.4, causal=True)
    for key in b:
        assert np.array_equal(a[key], b[key]), key


@pytest.mark.parametrize("causal", [False, True])
def test_gqa_global_identities(causal):
    q, k, v, do, uq, uk, uv = inputs(1, 6, 2, 19, 4, 6)
    tau = 0.5
    o = oracle.bob_gqa(q, k, v, do, uq, uk, uv, tau, causal=causal)
    ip = lambda a, b: float(np.sum(a * b))
    phi = ip(o["dQ"], uq) + ip(o["dK"], uk) + ip(o["dV"], uv)
    assert abs(ip(do, o["dOt"]) - phi) <= 1e-10 * (1 + abs(phi))                          # I1
    assert abs(ip(v, o["Vt"]) - (ip(o["dQ"], uq) + ip(o["dK"], uk))) <= 1e-10 * (1 + abs(phi))  # I2
    lhs = ip(q, o["Qt"]) - ip(k, o["Kt"])
    assert abs(lhs - (ip(o["dK"], uk) - ip(o["dQ"], uq))) <= 1e-10 * (1 + abs(phi))     # I3


GROUPING_MUTATIONS = {
    "key/value head h % Hkv instead of h // G": ("expand_kv", lambda X, G: np.tile(np.asarray(X, dtype=np.float64), (1, G, 1, 1))),
    "group sum keeps the first head only": ("group_sum", lambda X, G: np.asarray(X)[:, ::G].copy()),
    "group mean instead of sum": ("group_sum", lambda X, G: np.asarray(X).reshape((X.shape[0], X.shape[1] // G, G) + X.shape[2:]).mean(axis=2)),
}


@pytest.mark.parametrize("name", sorted(GROUPING_MUTATIONS))
def test_torch_pin_catches_grouping_mistakes(name, monkeypatch):
    x = inputs(1, 4, 2, 7, 3, 7)
    tau = 0.6
    tb = torch_gqa_bob(*x, tau, causal=False)
    attr, wrong = GROUPING_MUTATIONS[name]
    monkeypatch.setattr(bo, attr, wrong)
    out = bo.bob_gqa(*x, tau, causal=False)
    errs = [rel(out[key], tb[key]) for key in ("Qt", "Kt", "Vt", "dOt")]
    assert max(errs) > 1e-4, (name, errs)
