"""Pins for the float64 oracle, checked against what the paper and the
mathematics fix rather than against the oracle itself.

* library routines: scipy softmax / logsumexp for P, L, O (eq. 1);
* central finite differences (FD) of Phi (eq. 4) through an independently
  written first backward (one row at a time, explicit softmax Jacobian):
  every coordinate of every BoB output (eq. 5) at tiny N, d;
* FD of L and of O along (U_Q, U_K, U_V): alpha is the directional derivative
  of L, tilde-dO is the forward JVP of O;
* the Hessian symmetry <v, H u> = <u, H v> (Sec. 3.1: BoB of a gradient is
  an HVP);
* special cases: the forward-attention embedding of the lower-bound proof
  (App. D), U_Q = U_K = 0 (reduces to a first backward with V := U_V), N = 1;
* global identities that follow from homogeneity and shift invariance.
"""
import numpy as np
import pytest
from scipy.special import logsumexp, softmax

import oracle
from oracle import bob_oracle as bo

RNG = np.random.default_rng(12345)


def rand_inputs(n, d, rng=RNG, scale_qk=1.0):
    q = rng.standard_normal((n, d)) * scale_qk
    k = rng.standard_normal((n, d)) * scale_qk
    v, do, uq, uk, uv = (rng.standard_normal((n, d)) for _ in range(5))
    return q, k, v, do, uq, uk, uv


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def fd_grad(f, x, eps_rel=1e-5):
    """Central differences of scalar f at x, every coordinate."""
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        idx = it.multi_index
        h = eps_rel * (1.0 + abs(x[idx]))
        xp = x.copy(); xp[idx] += h
        xm = x.copy(); xm[idx] -= h
        g[idx] = (f(xp) - f(xm)) / (2 * h)
    return g


# ---------------------------------------------------------------- forward


@pytest.mark.parametrize("n,d", [(1, 4), (7, 3), (33, 16)])
def test_forward_matches_scipy(n, d):
    q, k, v, *_ = rand_inputs(n, d)
    tau = 1 / np.sqrt(d)
    O, L, P, S = bo.forward_head(q, k, v, tau)
    S_ref = tau * np.einsum("ia,ja->ij", q, k)
    np.testing.assert_allclose(L, logsumexp(S_ref, axis=1), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(P, softmax(S_ref, axis=1), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(O, softmax(S_ref, axis=1) @ v, rtol=1e-12, atol=1e-13)


def test_forward_large_logits_stable():
    q, k, v, *_ = rand_inputs(16, 8)
    O, L, P, _ = bo.forward_head(q * 40, k * 40, v, 1 / np.sqrt(8))
    assert np.isfinite(L).all() and np.isfinite(O).all()
    np.testing.assert_allclose(P.sum(1), 1.0, rtol=1e-13)


# ---------------------------------------------------------- first backward


@pytest.mark.parametrize("n,d", [(1, 2), (5, 3), (12, 8)])
def test_first_backward_matches_rowloop_and_D_identity(n, d):
    q, k, v, do, *_ = rand_inputs(n, d)
    tau = 0.7
    fb = bo.first_backward_head(q, k, v, do, tau)
    dq, dk, dv = bo.first_backward_rowloop(q, k, v, do, tau)
    assert rel(fb["dQ"], dq) < 1e-12 and rel(fb["dK"], dk) < 1e-12 and rel(fb["dV"], dv) < 1e-12
    # D_i = sum_j P_ij dP_ij = do_i . o_i (the identity stated after eq. 3)
    np.testing.assert_allclose(fb["D"], (do * fb["O"]).sum(1), rtol=1e-12, atol=1e-13)
    # shift invariance of softmax in K: sum_j dK_j = 0
    np.testing.assert_allclose(fb["dK"].sum(0), 0.0, atol=1e-12)


def test_first_backward_fd_of_loss():
    n, d = 5, 3
    q, k, v, do, *_ = rand_inputs(n, d)
    tau = 0.9

    def loss_q(x):
        return float((bo.forward_head(x, k, v, tau)[0] * do).sum())

    def loss_k(x):
        return float((bo.forward_head(q, x, v, tau)[0] * do).sum())

    def loss_v(x):
        return float((bo.forward_head(q, k, x, tau)[0] * do).sum())

    fb = bo.first_backward_head(q, k, v, do, tau)
    assert rel(fb["dQ"], fd_grad(loss_q, q)) < 1e-8
    assert rel(fb["dK"], fd_grad(loss_k, k)) < 1e-8
    assert rel(fb["dV"], fd_grad(loss_v, v)) < 1e-8


# ------------------------------------------------------------- BoB by FD


def bob_fd(q, k, v, do, uq, uk, uv, tau):
    """Gradient of Phi (eq. 4) by central FD through the row-loop first backward."""
    gq = fd_grad(lambda x: bo.phi_rowloop(x, k, v, do, uq, uk, uv, tau), q)
    gk = fd_grad(lambda x: bo.phi_rowloop(q, x, v, do, uq, uk, uv, tau), k)
    gv = fd_grad(lambda x: bo.phi_rowloop(q, k, x, do, uq, uk, uv, tau), v)
    gdo = fd_grad(lambda x: bo.phi_rowloop(q, k, v, x, uq, uk, uv, tau), do)
    return gq, gk, gv, gdo


@pytest.mark.parametrize("n,d", [(1, 1), (2, 1), (2, 2), (3, 4), (5, 2), (8, 8)])
def test_bob_every_coordinate_matches_fd(n, d):
    rng = np.random.default_rng(100 + 10 * n + d)
    args = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    out = bo.bob_head(*args, tau)
    gq, gk, gv, gdo = bob_fd(*args, tau)
    for name, fd in (("Qt", gq), ("Kt", gk), ("Vt", gv), ("dOt", gdo)):
        err = np.abs(out[name] - fd).max() / max(1.0, np.abs(fd).max())
        assert err < 1e-7, (name, err)


def test_bob_random_direction_fd_n64():
    rng = np.random.default_rng(7)
    n, d = 64, 16
    q, k, v, do, uq, uk, uv = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    out = bo.bob_head(q, k, v, do, uq, uk, uv, tau)
    # directional derivative of Phi along a random (dq, dk, dv, ddo)
    dirs = [rng.standard_normal((n, d)) for _ in range(4)]
    phi = lambda t: bo.phi_rowloop(q + t * dirs[0], k + t * dirs[1], v + t * dirs[2],
                                   do + t * dirs[3], uq, uk, uv, tau)
    h = 1e-5
    fd = (phi(h) - phi(-h)) / (2 * h)
    an = sum(float((o * w).sum()) for o, w in zip((out["Qt"], out["Kt"], out["Vt"], out["dOt"]), dirs))
    assert abs(fd - an) <= 1e-7 * max(1.0, abs(an))


# ---------------------------------------------------- row scalars, JVPs


def test_alpha_is_directional_derivative_of_L():
    rng = np.random.default_rng(3)
    n, d = 9, 5
    q, k, v, do, uq, uk, uv = rand_inputs(n, d, rng)
    tau = 0.45
    out = bo.bob_head(q, k, v, do, uq, uk, uv, tau)
    h = 1e-6
    Lp = bo.forward_head(q + h * uq, k + h * uk, v, tau)[1]
    Lm = bo.forward_head(q - h * uq, k - h * uk, v, tau)[1]
    np.testing.assert_allclose(out["alpha"], (Lp - Lm) / (2 * h), rtol=1e-7, atol=1e-8)


def test_dOt_is_forward_jvp_of_O_and_E_identity():
    rng = np.random.default_rng(4)
    n, d = 9, 5
    q, k, v, do, uq, uk, uv = rand_inputs(n, d, rng)
    tau = 0.45
    out = bo.bob_head(q, k, v, do, uq, uk, uv, tau)
    h = 1e-6
    Op = bo.forward_head(q + h * uq, k + h * uk, v + h * uv, tau)[0]
    Om = bo.forward_head(q - h * uq, k - h * uk, v - h * uv, tau)[0]
    jvp = (Op - Om) / (2 * h)
    np.testing.assert_allclose(out["dOt"], jvp, rtol=1e-7, atol=1e-8)
    # E_i = do_i . dOt_i - alpha_i D_i, with dOt pinned above, D = do . o and
    # alpha pinned by the L derivative; both sides use independent routes.
    O = bo.forward_head(q, k, v, tau)[0]
    D = (do * O).sum(1)
    np.testing.assert_allclose(out["E"], (do * jvp).sum(1) - out["alpha"] * D, rtol=1e-6, atol=1e-7)


def test_affine_fusion_matches_closed_form():
    rng = np.random.default_rng(5)
    for n, d in ((1, 3), (17, 8), (40, 16)):
        args = rand_inputs(n, d, rng)
        tau = 1 / np.sqrt(d)
        a = bo.bob_affine_head(*args, tau)
        c = bo.bob_head(*args, tau)
        for key in ("Qt", "dOt", "alpha", "E"):
            diff = np.linalg.norm(a[key] - c[key])
            assert diff <= 1e-12 * (1.0 + np.linalg.norm(c[key])), key


def test_threepass_route_matches_closed_form():
    """The three-pass control route (alpha first, then the delayed E
    correction) reaches the closed form of eqs. 6-7, dense and causal."""
    rng = np.random.default_rng(55)
    for n, d in ((1, 3), (17, 8), (40, 16)):
        for causal in (False, True):
            args = rand_inputs(n, d, rng)
            tau = 1 / np.sqrt(d)
            a = bo.bob_threepass_head(*args, tau, causal)
            c = bo.bob_head(*args, tau, causal)
            for key in ("Qt", "dOt", "alpha", "E"):
                diff = np.linalg.norm(a[key] - c[key])
                assert diff <= 1e-12 * (1.0 + np.linalg.norm(c[key])), (key, causal)


# ---------------------------------------------------------- symmetry


def test_hessian_symmetry():
    """<v, H u> = <u, H v> over the (Q, K, V) blocks (BoB of a gradient is an HVP)."""
    rng = np.random.default_rng(6)
    n, d = 24, 8
    q, k, v, do, *_ = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    u = [rng.standard_normal((n, d)) for _ in range(3)]
    w = [rng.standard_normal((n, d)) for _ in range(3)]
    hu = bo.bob_head(q, k, v, do, *u, tau)
    hw = bo.bob_head(q, k, v, do, *w, tau)
    a = sum(float((x * y).sum()) for x, y in zip(w, (hu["Qt"], hu["Kt"], hu["Vt"])))
    b = sum(float((x * y).sum()) for x, y in zip(u, (hw["Qt"], hw["Kt"], hw["Vt"])))
    assert abs(a - b) <= 1e-12 * max(1.0, abs(a))


# ------------------------------------------------------- special cases


def test_forward_embedding_instance():
    """App. D: V = dO = 0, U_Q = U_K = 0, U_V = W gives tilde-dO = softmax(tau Q K^T) W."""
    rng = np.random.default_rng(8)
    n, d = 20, 6
    q, k, w = (rng.standard_normal((n, d)) for _ in range(3))
    z = np.zeros((n, d))
    tau = 1 / np.sqrt(d)
    out = bo.bob_head(q, k, z, z, z, z, w, tau)
    np.testing.assert_allclose(out["dOt"], softmax(tau * q @ k.T, axis=1) @ w, rtol=1e-12, atol=1e-14)
    for key in ("Qt", "Kt", "Vt", "alpha", "E"):
        assert np.abs(out[key]).max() == 0.0, key


def test_zero_query_key_cotangents_reduce_to_first_backward():
    """U_Q = U_K = 0: (Qt, Kt) is the first backward (dQ, dK) of attention with
    values U_V and upstream dO; Vt = 0; dOt = P U_V."""
    rng = np.random.default_rng(9)
    n, d = 11, 4
    q, k, v, do, _, _, uv = rand_inputs(n, d, rng)
    z = np.zeros((n, d))
    tau = 0.6
    out = bo.bob_head(q, k, v, do, z, z, uv, tau)
    dq, dk, _ = bo.first_backward_rowloop(q, k, uv, do, tau)
    assert rel(out["Qt"], dq) < 1e-12 and rel(out["Kt"], dk) < 1e-12
    assert np.abs(out["Vt"]).max() == 0.0
    np.testing.assert_allclose(out["dOt"], softmax(tau * q @ k.T, axis=1) @ uv, rtol=1e-12, atol=1e-14)


def test_single_token():
    rng = np.random.default_rng(10)
    args = rand_inputs(1, 5, rng)
    out = bo.bob_head(*args, 0.3)
    for key in ("Qt", "Kt", "Vt"):
        assert np.abs(out[key]).max() < 1e-15, key
    np.testing.assert_allclose(out["dOt"], args[6], rtol=0, atol=1e-15)


# -------------------------------------------------- global identities


def global_identities(q, k, v, do, uq, uk, uv, out):
    """I1..I6: exact consequences of homogeneity / shift invariance of Phi."""
    ip = lambda a, b: float((a * b).sum())
    phi = ip(out["dQ"], uq) + ip(out["dK"], uk) + ip(out["dV"], uv)
    return {
        "I1": (ip(do, out["dOt"]), phi),                                   # Phi linear in dO
        "I2": (ip(v, out["Vt"]), ip(out["dQ"], uq) + ip(out["dK"], uk)),   # dQ, dK linear in V
        "I3": (ip(q, out["Qt"]) - ip(k, out["Kt"]),
               ip(out["dK"], uk) - ip(out["dQ"], uq)),                     # Q -> cQ, K -> K/c
        "I5": (np.abs(out["Kt"].sum(0)).max(), 0.0),                       # K -> K + 1c^T
        "I6": (np.abs(out["Vt"].sum(0)).max(), 0.0),                       # V -> V + 1c^T
    }


def test_global_identities():
    rng = np.random.default_rng(11)
    n, d = 50, 8
    args = rand_inputs(n, d, rng)
    out = bo.bob_head(*args, 1 / np.sqrt(d))
    scale = sum(np.linalg.norm(x) ** 2 for x in args)
    for name, (a, b) in global_identities(*args, out).items():
        assert abs(a - b) <= 1e-11 * scale, name


# ---------------------------------------- linearity and equivariance


def test_linearity_and_dO_structure():
    rng = np.random.default_rng(12)
    n, d = 13, 4
    q, k, v, do, uq, uk, uv = rand_inputs(n, d, rng)
    _, _, _, _, wq, wk, wv = rand_inputs(n, d, rng)
    tau = 0.5
    a = bo.bob_head(q, k, v, do, uq, uk, uv, tau)
    b = bo.bob_head(q, k, v, do, wq, wk, wv, tau)
    c = bo.bob_head(q, k, v, do, 2 * uq - wq, 2 * uk - wk, 2 * uv - wv, tau)
    for key in ("Qt", "Kt", "Vt", "dOt"):
        assert rel(c[key], 2 * a[key] - b[key]) < 1e-12, key
    # (Qt, Kt, Vt) are linear in dO; dOt does not depend on dO
    e = bo.bob_head(q, k, v, 3 * do, uq, uk, uv, tau)
    for key in ("Qt", "Kt", "Vt"):
        assert rel(e[key], 3 * a[key]) < 1e-12, key
    assert rel(e["dOt"], a["dOt"]) < 1e-12


def test_permutation_equivariance():
    rng = np.random.default_rng(13)
    n, d = 10, 3
    q, k, v, do, uq, uk, uv = rand_inputs(n, d, rng)
    tau = 0.8
    base = bo.bob_head(q, k, v, do, uq, uk, uv, tau)
    pk = rng.permutation(n)
    kp = bo.bob_head(q, k[pk], v[pk], do, uq, uk[pk], uv[pk], tau)
    assert rel(kp["Kt"], base["Kt"][pk]) < 1e-12 and rel(kp["Vt"], base["Vt"][pk]) < 1e-12
    assert rel(kp["Qt"], base["Qt"]) < 1e-12 and rel(kp["dOt"], base["dOt"]) < 1e-12
    pq = rng.permutation(n)
    qp = bo.bob_head(q[pq], k, v, do[pq], uq[pq], uk, uv, tau)
    assert rel(qp["Qt"], base["Qt"][pq]) < 1e-12 and rel(qp["dOt"], base["dOt"][pq]) < 1e-12
    assert rel(qp["Kt"], base["Kt"]) < 1e-12 and rel(qp["Vt"], base["Vt"]) < 1e-12


# --------------------------------------------- slabs and batched wrappers


def test_row_slab_matches_full():
    rng = np.random.default_rng(14)
    n, d = 70, 8
    args = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    full = bo.bob_head(*args, tau)
    rows = np.array([0, 3, 17, 69, 40])
    part = bo.bob_rows(*args, tau, rows)
    for key in ("Qt", "dOt", "alpha", "E", "O", "L", "D", "dQ"):
        assert rel(part[key], full[key][rows]) < 1e-13, key


def test_batched_wrappers_are_per_head():
    rng = np.random.default_rng(15)
    B, H, n, d = 2, 3, 9, 4
    mats = [rng.standard_normal((B, H, n, d)) for _ in range(7)]
    tau = 0.5
    out = oracle.bob(*mats, tau)
    for b in range(B):
        for h in range(H):
            ref = bo.bob_head(*[m[b, h] for m in mats], tau)
            for key in ("Qt", "Kt", "Vt", "dOt", "alpha", "E", "L", "D"):
                assert rel(out[key][b, h], ref[key]) < 1e-14, key
    fw = oracle.forward(*mats[:3], tau)
    assert fw["O"].shape == (B, H, n, d) and fw["L"].shape == (B, H, n)


# ------------------------------------------------------------- golden file


def test_golden_tiny_case_unchanged():
    """tests/golden/bob_tiny_n5_d3.json was written by tests/golden/make_golden.py
    (oracle only); its inputs are stored in the file itself."""
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "bob_tiny_n5_d3.json")
    doc = json.load(open(path))
    args = [np.array(doc["inputs"][n]) for n in ("Q", "K", "V", "dO", "UQ", "UK", "UV")]
    out = bo.bob_head(*args, doc["tau"])
    for key, val in doc["outputs"].items():
        np.testing.assert_allclose(out[key], np.array(val), rtol=1e-13, atol=1e-14)


def test_column_slices_match_full():
    """bob_cols with row scalars from row_scalars (slabbed bob_rows) gives the
    same Kt, Vt, dK, dV columns as the full materialised bob_head."""
    rng = np.random.default_rng(16)
    n, d = 90, 8
    args = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    full = bo.bob_head(*args, tau)
    rs = bo.row_scalars(*args, tau, slab=32)
    for key in ("alpha", "E", "L", "D"):
        assert rel(rs[key], full[key]) < 1e-13, key
    cols = np.array([0, 5, 31, 32, 89])
    part = bo.bob_cols(*args, tau, cols, rs["alpha"], rs["E"], rs["L"], rs["D"])
    for key in ("Kt", "Vt", "dK", "dV"):
        assert rel(part[key], full[key][cols]) < 1e-13, key


@pytest.mark.parametrize("causal", [False, True])
def test_threaded_row_scalars_match_full(causal):
    """row_scalars over uneven slabs in several threads gives the full
    materialised bob_head's alpha, E, L, D, and reports every row once."""
    rng = np.random.default_rng(17)
    n, d = 101, 8
    args = rand_inputs(n, d, rng)
    tau = 1 / np.sqrt(d)
    full = bo.bob_head(*args, tau, causal=causal)
    seen = []
    rs = bo.row_scalars(*args, tau, slab=7, causal=causal, workers=4, progress=lambda k, m: seen.append((k, m)))
    for key in ("alpha", "E", "L", "D"):
        assert rel(rs[key], full[key]) < 1e-13, key
    assert sorted(k for k, _ in seen)[-1] == n and all(m == n for _, m in seen) and len(seen) == -(-n // 7)
