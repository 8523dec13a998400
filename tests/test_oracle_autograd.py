"""Pin of the oracle's BoB against torch's own double backward.

PyTorch's autograd, run twice in float64 on a plain softmax-attention
forward written with tensor primitives (matmul, masked_fill, softmax), is an
implementation of the same map that shares nothing with the oracle: the
first backward and the backward of that backward are derived by the
autograd engine rather than from eqs. 2-7.  With dQ, dK, dV = grad of
<O, dO> (create_graph) and Phi = <dQ, U_Q> + <dK, U_K> + <dV, U_V> (eq. 4),
grad(Phi) with respect to (Q, K, V, dO) must equal the oracle's
(Qt, Kt, Vt, dOt) (eq. 5) to float64 round-off, dense and causal, and the
first backward must equal the oracle's dQ, dK, dV.  CPU only."""
import numpy as np
import pytest
import torch

import oracle

TOL = 1e-11


def torch_bob(q, k, v, do, uq, uk, uv, tau, causal):
    Q, K, V, dO = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (q, k, v, do))
    UQ, UK, UV = (torch.tensor(a, dtype=torch.float64) for a in (uq, uk, uv))
    S = tau * (Q @ K.T)
    if causal:
        n = S.shape[0]
        mask = torch.ones(n, n, dtype=torch.bool).triu(1)
        S = S.masked_fill(mask, float("-inf"))
    O = torch.softmax(S, dim=-1) @ V
    dQ, dK, dV = torch.autograd.grad(O, (Q, K, V), grad_outputs=dO, create_graph=True)
    phi = (dQ * UQ).sum() + (dK * UK).sum() + (dV * UV).sum()
    Qt, Kt, Vt, dOt = torch.autograd.grad(phi, (Q, K, V, dO))
    first = {"dQ": dQ.detach().numpy(), "dK": dK.detach().numpy(), "dV": dV.detach().numpy()}
    second = {"Qt": Qt.numpy(), "Kt": Kt.numpy(), "Vt": Vt.numpy(), "dOt": dOt.numpy()}
    return first, second


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


@pytest.mark.parametrize("n,d,causal,seed", [(37, 8, False, 1), (37, 8, True, 2), (5, 3, False, 3),
                                             (64, 16, True, 4), (1, 4, False, 5)])
def test_oracle_matches_torch_double_backward(n, d, causal, seed):
    rng = np.random.default_rng(seed)
    q, k, v, do, uq, uk, uv = (rng.standard_normal((n, d)) for _ in range(7))
    tau = 1.0 / np.sqrt(d)
    ref = oracle.bob_head(q, k, v, do, uq, uk, uv, tau, causal=causal)
    first, second = torch_bob(q, k, v, do, uq, uk, uv, tau, causal)
    for name, val in {**first, **second}.items():
        err = rel(ref[name], val) if np.linalg.norm(val) > 0 else np.linalg.norm(ref[name])
        assert err <= TOL, (name, err)


def test_affine_route_matches_torch_double_backward():
    """The six-accumulator route of Prop. 3.1 against the same autograd result."""
    rng = np.random.default_rng(6)
    n, d = 29, 8
    q, k, v, do, uq, uk, uv = (rng.standard_normal((n, d)) for _ in range(7))
    tau = 0.3
    _, second = torch_bob(q, k, v, do, uq, uk, uv, tau, causal=True)
    aff = oracle.bob_affine_head(q, k, v, do, uq, uk, uv, tau, causal=True)
    for name in ("Qt", "dOt"):
        assert rel(aff[name], second[name]) <= TOL, name
