"""Pins for the causal-mask path of the oracle (M_mask = -inf above the
diagonal, Sec. 2).  The same independent pins as the dense case, with the
row-loop first backward restricted to keys 0..i, plus causal-only facts."""
import numpy as np
import pytest
from scipy.special import softmax

from oracle import bob_oracle as bo
from tests.test_oracle_pins import fd_grad, global_identities, rand_inputs, rel


def bob_fd_causal(q, k, v, do, uq, uk, uv, tau):
    f = lambda *m: bo.phi_rowloop(*m, uq, uk, uv, tau, causal=True)
    return (fd_grad(lambda x: f(x, k, v, do), q), fd_grad(lambda x: f(q, x, v, do), k),
            fd_grad(lambda x: f(q, k, x, do), v), fd_grad(lambda x: f(q, k, v, x), do))


@pytest.mark.parametrize("n,d", [(1, 2), (2, 1), (3, 4), (5, 2), (8, 8)])
def test_causal_bob_every_coordinate_matches_fd(n, d):
    rng = np.random.default_rng(300 + 10 * n + d)
    args = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    out = bo.bob_head(*args, tau, causal=True)
    for name, g in zip(("Qt", "Kt", "Vt", "dOt"), bob_fd_causal(*args, tau)):
        err = np.abs(out[name] - g).max() / max(1.0, np.abs(g).max())
        assert err < 1e-7, (name, err)


def test_causal_forward_and_first_backward():
    rng = np.random.default_rng(31)
    n, d = 13, 4
    q, k, v, do, *_ = rand_inputs(n, d, rng)
    tau = 0.6
    S = tau * q @ k.T
    S[np.triu_indices(n, 1)] = -np.inf
    O, L, P, _ = bo.forward_head(q, k, v, tau, causal=True)
    np.testing.assert_allclose(P, softmax(S, axis=1), rtol=1e-12, atol=1e-15)
    assert np.all(P[np.triu_indices(n, 1)] == 0.0)
    fb = bo.first_backward_head(q, k, v, do, tau, causal=True)
    dq, dk, dv = bo.first_backward_rowloop(q, k, v, do, tau, causal=True)
    assert rel(fb["dQ"], dq) < 1e-12 and rel(fb["dK"], dk) < 1e-12 and rel(fb["dV"], dv) < 1e-12


def test_causal_first_row_and_prefix():
    """Row 0 sees only key 0, so Qt_0 = 0 and dOt_0 = U_V[0]; and rows < m depend
    only on the first m rows of every input (a prefix of a causal problem)."""
    rng = np.random.default_rng(32)
    n, d, m = 20, 6, 9
    args = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    full = bo.bob_head(*args, tau, causal=True)
    assert np.abs(full["Qt"][0]).max() < 1e-14
    np.testing.assert_allclose(full["dOt"][0], args[6][0], rtol=0, atol=1e-14)
    pre = bo.bob_head(*[a[:m] for a in args], tau, causal=True)
    for key in ("Qt", "dOt", "alpha", "E", "L", "D"):
        assert rel(pre[key], full[key][:m]) < 1e-12, key


def test_causal_symmetry_identities_and_slices():
    rng = np.random.default_rng(33)
    n, d = 40, 8
    q, k, v, do, uq, uk, uv = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    w = [rng.standard_normal((n, d)) for _ in range(3)]
    hu = bo.bob_head(q, k, v, do, uq, uk, uv, tau, causal=True)
    hw = bo.bob_head(q, k, v, do, *w, tau, causal=True)
    a = sum(float((x * y).sum()) for x, y in zip(w, (hu["Qt"], hu["Kt"], hu["Vt"])))
    b = sum(float((x * y).sum()) for x, y in zip((uq, uk, uv), (hw["Qt"], hw["Kt"], hw["Vt"])))
    assert abs(a - b) <= 1e-12 * max(1.0, abs(a))
    scale = sum(np.linalg.norm(x) ** 2 for x in (q, k, v, do, uq, uk, uv))
    for name, (x, y) in global_identities(q, k, v, do, uq, uk, uv, hu).items():
        assert abs(x - y) <= 1e-11 * scale, name
    aff = bo.bob_affine_head(q, k, v, do, uq, uk, uv, tau, causal=True)
    for key in ("Qt", "dOt", "alpha", "E"):
        assert rel(aff[key], hu[key]) < 1e-12, key
    rows = np.array([0, 7, 39])
    part = bo.bob_rows(q, k, v, do, uq, uk, uv, tau, rows, causal=True)
    for key in ("Qt", "dOt", "alpha", "E", "L", "D", "dQ"):
        assert rel(part[key], hu[key][rows]) < 1e-12, key
    rs = bo.row_scalars(q, k, v, do, uq, uk, uv, tau, slab=16, causal=True)
    cols = np.array([0, 20, 39])
    pc = bo.bob_cols(q, k, v, do, uq, uk, uv, tau, cols, rs["alpha"], rs["E"], rs["L"], rs["D"], causal=True)
    for key in ("Kt", "Vt", "dK", "dV"):
        assert rel(pc[key], hu[key][cols]) < 1e-12, key


def test_causal_forward_embedding():
    rng = np.random.default_rng(34)
    n, d = 15, 5
    q, k, wv = (rng.standard_normal((n, d)) for _ in range(3))
    z = np.zeros((n, d))
    tau = 0.4
    out = bo.bob_head(q, k, z, z, z, z, wv, tau, causal=True)
    S = tau * q @ k.T
    S[np.triu_indices(n, 1)] = -np.inf
    np.testing.assert_allclose(out["dOt"], softmax(S, axis=1) @ wv, rtol=1e-12, atol=1e-14)
