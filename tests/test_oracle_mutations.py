"""Planted mistakes in the oracle (on the CPU) must be caught by its pins.

Each case replaces one named step of the oracle with a plausible wrong
version (a dropped term, a flipped sign, a transposed operand, a wrong
index) and checks that the finite-difference pin of Phi (eq. 4) no longer
agrees.  This shows the pins are sharp enough to catch such slips.
"""
import numpy as np
import pytest

from oracle import bob_oracle as bo
from tests.test_oracle_pins import bob_fd, rand_inputs

MUTATIONS = {
    "F drops Q U_K^T": ("F_of", lambda q, k, uq, uk, tau: tau * (uq @ k.T)),
    "F transposed operand": ("F_of", lambda q, k, uq, uk, tau: tau * (k @ uq.T + uk @ q.T)),
    "C transposed": ("C_of", lambda do, uv: uv @ do.T),
    "alpha without P": ("alpha_of", lambda P, F: F.sum(axis=-1)),
    "Ptilde alpha sign": ("Ptilde_of", lambda C, F, dP, D, a: C + F * (dP - D[:, None]) + a[:, None] * dP),
    "Ptilde drops C": ("Ptilde_of", lambda C, F, dP, D, a: F * (dP - D[:, None]) - a[:, None] * dP),
    "Stilde drops E": ("Stilde_of", lambda P, Pt, E: P * Pt),
    "E column sum": ("E_of", lambda P, Pt: np.broadcast_to((P * Pt).sum(axis=0), P.shape[:1]).copy()),
    "dS D sign": ("dS_of", lambda P, dP, D: P * (dP + D[:, None])),
    "scores missing tau": ("scores", lambda q, k, tau, *a, **kw: q @ k.T),
    "dP transposed": ("dP_of", lambda do, v: v @ do.T),
    "row D from P only": ("row_D", lambda P, dP: dP.sum(axis=-1)),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_fd_pin_catches_planted_mistake(name, monkeypatch):
    attr, wrong = MUTATIONS[name]
    rng = np.random.default_rng(77)
    n, d = 4, 3
    args = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    fd = bob_fd(*args, tau)                    # computed before the mutation
    monkeypatch.setattr(bo, attr, wrong)
    out = bo.bob_head(*args, tau)
    errs = [np.abs(out[key] - g).max() / max(1.0, np.abs(g).max())
            for key, g in zip(("Qt", "Kt", "Vt", "dOt"), fd)]
    assert max(errs) > 1e-4, (name, errs)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_torch_double_backward_pin_catches_planted_mistake(name, monkeypatch):
    """The same planted mistakes also break agreement with torch's own double
    backward (tests/test_oracle_autograd.py)."""
    from tests.test_oracle_autograd import torch_bob
    attr, wrong = MUTATIONS[name]
    rng = np.random.default_rng(78)
    n, d = 6, 4
    args = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    _, ref = torch_bob(*args, tau, causal=False)   # computed before the mutation
    monkeypatch.setattr(bo, attr, wrong)
    out = bo.bob_head(*args, tau)
    errs = [np.abs(out[key] - ref[key]).max() / max(1.0, np.abs(ref[key]).max())
            for key in ("Qt", "Kt", "Vt", "dOt")]
    assert max(errs) > 1e-4, (name, errs)
