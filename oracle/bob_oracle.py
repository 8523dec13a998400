"""Plain float64 oracle for attention BoB (test infrastructure only).

Parity pins live in the CPU test suite; see the module docstring of
``oracle`` for who may use this file.  Notation follows the paper:
tau is the softmax scale, U_Q, U_K, U_V are the cotangents on the
first-backward outputs (dQ, dK, dV), and the BoB outputs are
Qt, Kt, Vt, dOt (the paper's tilde-Q, tilde-K, tilde-V, tilde-dO).

Layout: every matrix argument is [..., N, d] (any leading batch/head
dims); row vectors (L, D, alpha, E) are [..., N].  The *_head functions
take a single head ([N, d]) and are the definitions; the batched wrappers
loop over leading dims.

Each step is a small named function so a reader can check it against the
paper line by line, and so the CPU tests can perturb a single step to show
that the pins catch the mistake.
"""
import numpy as np

# --------------------------------------------------------------------------
# Forward attention (Sec. 2, eq. 1; L as defined in the FlashAttention
# paragraph of Sec. 2 and in the notation table, App. "Notation").
# --------------------------------------------------------------------------


def scores(q, k, tau, causal=False, q_idx=None, k_idx=None):
    """S = tau * Q K^T + M_mask (eq. 1).

    Without a mask every key is valid.  With causal=True, M_mask is -inf
    where the key index exceeds the query index (the causal pattern named in
    Sec. 2), so P is zero there and every row sum runs over the valid set
    V_i = {j <= i}.  q_idx / k_idx give the absolute indices of the rows of
    q and k when they are slices (default: 0..n-1).
    """
    S = tau * (q @ k.T)
    if causal:
        qi = np.arange(q.shape[0]) if q_idx is None else np.asarray(q_idx)
        kj = np.arange(k.shape[0]) if k_idx is None else np.asarray(k_idx)
        S = np.where(kj[None, :] <= qi[:, None], S, -np.inf)
    return S


def log_normalizer(S):
    """L_i = log sum_j exp(S_ij), computed max-subtracted."""
    m = S.max(axis=-1)
    return m + np.log(np.exp(S - m[:, None]).sum(axis=-1))


def probabilities(S, L):
    """P_ij = exp(S_ij - L_i): row softmax recomputed from the saved L."""
    return np.exp(S - L[:, None])


def forward_head(q, k, v, tau, causal=False):
    """Eq. 1: S = tau Q K^T (+ mask), P = softmax(S), O = P V; plus L.

    Returns (O, L, P, S).
    """
    S = scores(q, k, tau, causal)
    L = log_normalizer(S)
    P = probabilities(S, L)
    O = P @ v
    return O, L, P, S


# --------------------------------------------------------------------------
# First backward (Sec. 2, eqs. 2-3).
# --------------------------------------------------------------------------


def dP_of(do, v):
    """dP = dO V^T (eq. 2)."""
    return do @ v.T


def row_D(P, dP):
    """D_i = sum_j P_ij dP_ij (the row scalar after eq. 3)."""
    return (P * dP).sum(axis=-1)


def dS_of(P, dP, D):
    """dS_ij = P_ij (dP_ij - D_i) (eq. 2)."""
    return P * (dP - D[:, None])


def first_backward_head(q, k, v, do, tau, causal=False):
    """Eqs. 2-3 on one head, materialised.

    Returns a dict with O, L, P, S, dP, D, dS, dQ, dK, dV.
    """
    O, L, P, S = forward_head(q, k, v, tau, causal)
    dP = dP_of(do, v)
    D = row_D(P, dP)
    dS = dS_of(P, dP, D)
    return dict(
        O=O, L=L, P=P, S=S, dP=dP, D=D, dS=dS,
        dQ=tau * (dS @ k),          # eq. 3
        dK=tau * (dS.T @ q),        # eq. 3
        dV=P.T @ do,                # eq. 2
    )


# --------------------------------------------------------------------------
# BoB closed form (Sec. 3.2 eqs. 6-7 with the definitions that follow them;
# the same list appears as "Final assembled identities" in App. A).
# --------------------------------------------------------------------------


def F_of(q, k, uq, uk, tau):
    """F = tau (U_Q K^T + Q U_K^T): BoB gradient at dS (App. A step 1)."""
    return tau * (uq @ k.T + q @ uk.T)


def C_of(do, uv):
    """C = dO U_V^T: contribution to tilde-P from the dV child (App. A step 4)."""
    return do @ uv.T


def alpha_of(P, F):
    """alpha_i = sum_j P_ij F_ij (App. A step 2)."""
    return (P * F).sum(axis=-1)


def Ptilde_of(C, F, dP, D, alpha):
    """tilde-P_ij = C_ij + F_ij (dP_ij - D_i) - alpha_i dP_ij (App. A step 5)."""
    return C + F * (dP - D[:, None]) - alpha[:, None] * dP


def E_of(P, Pt):
    """E_i = sum_j P_ij tilde-P_ij (App. A step 6)."""
    return (P * Pt).sum(axis=-1)


def Stilde_of(P, Pt, E):
    """tilde-S = P (.) (tilde-P - E 1^T) (App. A step 6)."""
    return P * (Pt - E[:, None])


def bob_head(q, k, v, do, uq, uk, uv, tau, causal=False):
    """All four BoB outputs on one head, eqs. 6-7, fully materialised.

    With causal=True the masked entries have P = 0, so every sum runs over
    the valid columns of its row (Sec. 2 and App. A).  Returns a dict with
    Qt, Kt, Vt, dOt, alpha, E and the producer state O, L, D, dQ, dK, dV.
    """
    fb = first_backward_head(q, k, v, do, tau, causal)
    P, dP, D, dS = fb["P"], fb["dP"], fb["D"], fb["dS"]
    F = F_of(q, k, uq, uk, tau)
    alpha = alpha_of(P, F)
    h = F - alpha[:, None]
    C = C_of(do, uv)
    Pt = Ptilde_of(C, F, dP, D, alpha)
    E = E_of(P, Pt)
    St = Stilde_of(P, Pt, E)
    Ph = P * h
    return dict(
        Qt=tau * (St @ k + dS @ uk),        # eq. 6
        Kt=tau * (St.T @ q + dS.T @ uq),    # eq. 6
        Vt=Ph.T @ do,                       # eq. 7
        dOt=P @ uv + Ph @ v,                # eq. 7
        alpha=alpha, E=E,
        O=fb["O"], L=fb["L"], D=D, dQ=fb["dQ"], dK=fb["dK"], dV=fb["dV"],
    )


def bob_affine_head(q, k, v, do, uq, uk, uv, tau, causal=False):
    """Row-owned outputs through the affine fusion of Prop. 3.1 (eq. 8).

    The six row accumulators are the sums named in the proof of Prop. 3.1
    (App. B): alpha, E0 = sum P Pt0, dOt0 = P U_V + (P F) V,
    Omega = (P Pt0) K + (P (dP - D)) U_K, B = P K, R = (P dP) K, with the
    alpha-free Pt0 = C + F (dP - D).  The corrections of eq. 8 then give
    E, dOt and Qt.  Here the sums run over the whole row at once (no tiling),
    so this is a second route to the same numbers, not the tiled schedule.
    """
    O, L, P, _ = forward_head(q, k, v, tau, causal)
    dP = dP_of(do, v)
    D = row_D(P, dP)
    F = F_of(q, k, uq, uk, tau)
    C = C_of(do, uv)
    Pt0 = C + F * (dP - D[:, None])
    alpha = (P * F).sum(axis=-1)
    E0 = (P * Pt0).sum(axis=-1)
    dOt0 = P @ uv + (P * F) @ v
    Omega = (P * Pt0) @ k + (P * (dP - D[:, None])) @ uk
    Bacc = P @ k
    R = (P * dP) @ k
    E = E0 - alpha * D
    dOt = dOt0 - alpha[:, None] * O
    Qt = tau * (Omega - alpha[:, None] * R - E[:, None] * Bacc)
    return dict(Qt=Qt, dOt=dOt, alpha=alpha, E=E, E0=E0)


def bob_threepass_head(q, k, v, do, uq, uk, uv, tau, causal=False):
    """Row-owned outputs through the three-pass control schedule (App.
    "Three-pass versus two-pass"; the three-pass overlay figure of App.
    "Dependency graphs").

    Its first sweep forms only alpha = sum_j P F.  Its second sweep, with
    alpha known, forms Pt = C + F (dP - D) - alpha dP and h = F - alpha
    directly and keeps one delayed correction: it accumulates
    E = sum_j P Pt, Omega' = (P Pt) K + dS U_K and B = P K, then
    Qt = tau (Omega' - E B) because S~ = P (Pt - E); dOt = P U_V + (P h) V.
    (Its third sweep is the column pass shared with the two-pass schedule.)
    Whole rows at once: a further route to the same numbers, not a tiling.
    """
    O, L, P, _ = forward_head(q, k, v, tau, causal)
    dP = dP_of(do, v)
    D = row_D(P, dP)
    F = F_of(q, k, uq, uk, tau)
    C = C_of(do, uv)
    # sweep 1
    alpha = (P * F).sum(axis=-1)
    # sweep 2
    Pt = C + F * (dP - D[:, None]) - alpha[:, None] * dP
    h = F - alpha[:, None]
    E = (P * Pt).sum(axis=-1)
    OmegaP = (P * Pt) @ k + (P * (dP - D[:, None])) @ uk
    Bacc = P @ k
    Qt = tau * (OmegaP - E[:, None] * Bacc)
    dOt = P @ uv + (P * h) @ v
    return dict(Qt=Qt, dOt=dOt, alpha=alpha, E=E)


# --------------------------------------------------------------------------
# An independently written first backward g(Q, K, V, dO) = (dQ, dK, dV):
# one query row at a time, the softmax Jacobian written out as
# diag(p) - p p^T (App. A step 6 derives it by the quotient rule).
# It shares no helper with the functions above and exists so that finite
# differences of Phi = <dQ,U_Q> + <dK,U_K> + <dV,U_V> (eq. 4) give an
# independent check of every BoB output (eq. 5).
# --------------------------------------------------------------------------


def first_backward_rowloop(q, k, v, do, tau, causal=False):
    n, d = q.shape
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for i in range(n):
        m = i + 1 if causal else n              # row i sees keys 0..m-1
        s = np.array([tau * float(np.dot(q[i], k[j])) for j in range(m)])
        e = np.exp(s - s.max())
        p = e / e.sum()
        grad_p = v[:m] @ do[i]                  # d<o_i, do_i>/dp_j = v_j . do_i
        jac = np.diag(p) - np.outer(p, p)       # dp/ds for one softmax row
        grad_s = jac.T @ grad_p
        dq[i] = tau * (grad_s @ k[:m])
        dk[:m] += tau * np.outer(grad_s, q[i])
        dv[:m] += np.outer(p, do[i])
    return dq, dk, dv


def phi_rowloop(q, k, v, do, uq, uk, uv, tau, causal=False):
    """Phi of eq. 4 evaluated through the independent first backward."""
    dq, dk, dv = first_backward_rowloop(q, k, v, do, tau, causal)
    return float((dq * uq).sum() + (dk * uk).sum() + (dv * uv).sum())


# --------------------------------------------------------------------------
# Batched wrappers: leading dims are independent heads (Sec. 2, "the analysis
# extends naturally to multiple heads").
# --------------------------------------------------------------------------


def _heads(x):
    return x.reshape((-1,) + x.shape[-2:])


def _batched(fn, keys, shapes_from, *mats, tau, causal=False):
    lead = shapes_from.shape[:-2]
    flat = [_heads(np.asarray(m, dtype=np.float64)) for m in mats]
    outs = [fn(*[m[h] for m in flat], tau, causal) for h in range(flat[0].shape[0])]
    res = {}
    for key in keys:
        arr = np.stack([o[key] for o in outs])
        res[key] = arr.reshape(lead + arr.shape[1:])
    return res


def forward(Q, K, V, tau, causal=False):
    """Batched eq. 1: returns dict(O, L)."""
    def f(q, k, v, t, c):
        O, L, _, _ = forward_head(q, k, v, t, c)
        return dict(O=O, L=L)
    return _batched(f, ("O", "L"), Q, Q, K, V, tau=tau, causal=causal)


def first_backward(Q, K, V, dO, tau, causal=False):
    """Batched eqs. 1-3: returns dict(O, L, D, dQ, dK, dV)."""
    keys = ("O", "L", "D", "dQ", "dK", "dV")
    return _batched(first_backward_head, keys, Q, Q, K, V, dO, tau=tau, causal=causal)


def bob(Q, K, V, dO, UQ, UK, UV, tau, causal=False):
    """Batched BoB (eqs. 6-7): dict(Qt, Kt, Vt, dOt, alpha, E, O, L, D, dQ, dK, dV)."""
    keys = ("Qt", "Kt", "Vt", "dOt", "alpha", "E", "O", "L", "D", "dQ", "dK", "dV")
    return _batched(bob_head, keys, Q, Q, K, V, dO, UQ, UK, UV, tau=tau, causal=causal)


def bob_threepass(Q, K, V, dO, UQ, UK, UV, tau, causal=False):
    """Batched three-pass control route: dict(Qt, dOt, alpha, E)."""
    keys = ("Qt", "dOt", "alpha", "E")
    return _batched(bob_threepass_head, keys, Q, Q, K, V, dO, UQ, UK, UV, tau=tau, causal=causal)


def bob_affine(Q, K, V, dO, UQ, UK, UV, tau, causal=False):
    """Batched Prop. 3.1 route: dict(Qt, dOt, alpha, E, E0)."""
    keys = ("Qt", "dOt", "alpha", "E", "E0")
    return _batched(bob_affine_head, keys, Q, Q, K, V, dO, UQ, UK, UV, tau=tau, causal=causal)


# --------------------------------------------------------------------------
# Grouped-query attention (the extension named in the paper's limitations):
# Hq query heads share Hkv key/value heads, G = Hq / Hkv, and query head h of a
# batch attends with key/value head h // G.  The first-backward dK, dV of a
# key/value head are the sums of its G query heads' contributions, so
# <dK, U_K> + <dV, U_V> splits into one term per query head with the shared
# U_K, U_V, and Phi (eq. 4) is the multi-head Phi with K, V, U_K, U_V repeated
# per query head.  Hence Qt, dOt, alpha, E are the single-head definitions of
# each query head, and Kt, Vt (like dK, dV) are summed over each group.
# --------------------------------------------------------------------------


def expand_kv(X, G):
    """[B, Hkv, N, d] -> [B, Hkv * G, N, d]; query head h reads head h // G."""
    return np.repeat(np.asarray(X, dtype=np.float64), G, axis=1)


def group_sum(X, G):
    """[B, Hkv * G, ...] -> [B, Hkv, ...]: sum over each group of G heads."""
    X = np.asarray(X, dtype=np.float64)
    return X.reshape((X.shape[0], X.shape[1] // G, G) + X.shape[2:]).sum(axis=2)


def bob_gqa(Q, K, V, dO, UQ, UK, UV, tau, causal=False):
    """BoB with grouped key/value heads: Q, dO, U_Q are [B, Hq, N, d] and
    K, V, U_K, U_V are [B, Hkv, N, d] with Hq a multiple of Hkv.  Returns the
    keys of `bob`, with Kt, Vt, dK, dV of shape [B, Hkv, N, d]."""
    Hq, Hkv = Q.shape[1], K.shape[1]
    assert Hkv >= 1 and Hq % Hkv == 0, (Hq, Hkv)
    G = Hq // Hkv
    out = bob(Q, expand_kv(K, G), expand_kv(V, G), dO, UQ, expand_kv(UK, G), expand_kv(UV, G), tau, causal=causal)
    for key in ("Kt", "Vt", "dK", "dV"):
        out[key] = group_sum(out[key], G)
    return out


def bob_rows(q, k, v, do, uq, uk, uv, tau, rows, causal=False):
    """Row-owned outputs of one head restricted to the query rows `rows`.

    Every row-owned quantity (Qt, dOt, alpha, E, O, L, D, dQ) of row i depends
    only on row i of the N x N matrices (Sec. 3.2: each is a sum over the
    columns of one fixed row), so the same definitions applied to a slab of query rows
    give exactly those rows.  Used for large N, where the full N x N matrices
    do not fit.
    """
    rows = np.asarray(rows)
    qi, doi, uqi = q[rows], do[rows], uq[rows]
    S = scores(qi, k, tau, causal, q_idx=rows)
    L = log_normalizer(S)
    P = probabilities(S, L)
    O = P @ v
    dP = dP_of(doi, v)
    D = row_D(P, dP)
    dS = dS_of(P, dP, D)
    F = F_of(qi, k, uqi, uk, tau)
    alpha = alpha_of(P, F)
    h = F - alpha[:, None]
    C = C_of(doi, uv)
    Pt = Ptilde_of(C, F, dP, D, alpha)
    E = E_of(P, Pt)
    St = Stilde_of(P, Pt, E)
    return dict(
        Qt=tau * (St @ k + dS @ uk),
        dOt=P @ uv + (P * h) @ v,
        alpha=alpha, E=E, O=O, L=L, D=D, dQ=tau * (dS @ k),
    )


def row_scalars_slab(q, k, v, do, uq, uk, uv, tau, rows, causal=False):
    """L, D, alpha, E of one head at the query rows `rows` only.

    The same step functions as bob_rows (each row scalar is a sum over the
    columns of one fixed row, Sec. 3.2), without the row-owned matrix outputs
    that bob_rows also forms."""
    rows = np.asarray(rows)
    qi, doi, uqi = q[rows], do[rows], uq[rows]
    S = scores(qi, k, tau, causal, q_idx=rows)
    L = log_normalizer(S)
    P = probabilities(S, L)
    del S
    dP = dP_of(doi, v)
    D = row_D(P, dP)
    F = F_of(qi, k, uqi, uk, tau)
    alpha = alpha_of(P, F)
    C = C_of(doi, uv)
    Pt = Ptilde_of(C, F, dP, D, alpha)
    E = E_of(P, Pt)
    return dict(alpha=alpha, E=E, L=L, D=D)


def row_scalars(q, k, v, do, uq, uk, uv, tau, slab=1024, causal=False, workers=1, progress=None):
    """alpha, E, L, D for every query row of one head, computed slab by slab
    with row_scalars_slab (row-owned, so slabs are exact).

    workers > 1 runs the slabs in that many threads (NumPy releases the GIL
    inside its array operations; BLAS is held to one thread per slab meanwhile).
    Slabs and threads change nothing but the BLAS's summation order.
    progress, if given, is called as progress(rows_done, n) after each slab."""
    import threading
    n = q.shape[0]
    out = {key: np.empty(n) for key in ("alpha", "E", "L", "D")}
    starts = list(range(0, n, slab))
    done = [0]
    lock = threading.Lock()

    def one(r0):
        rows = np.arange(r0, min(n, r0 + slab))
        part = row_scalars_slab(q, k, v, do, uq, uk, uv, tau, rows, causal)
        for key in out:
            out[key][rows] = part[key]
        if progress is not None:
            with lock:
                done[0] += len(rows)
                progress(done[0], n)

    if workers <= 1:
        for r0 in starts:
            one(r0)
        return out
    from concurrent.futures import ThreadPoolExecutor
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=1, user_api="blas"), ThreadPoolExecutor(max_workers=workers) as pool:
        for fut in [pool.submit(one, r0) for r0 in starts]:
            fut.result()
    return out


def bob_cols(q, k, v, do, uq, uk, uv, tau, cols, alpha, E, L, D, causal=False):
    """Column-owned outputs of one head (Kt, Vt, and the producer's dK, dV) at
    the key rows `cols`.

    Column j sums over every query row i (Sec. 3.2: Kt and Vt are sums over
    the rows of one fixed column), so the row scalars alpha, E, L, D of all rows are
    inputs here; callers compute them with row_scalars() from this module.
    The per-tile quantities follow the same definitions as bob_head, taken on
    the N x |cols| slice of the attention matrices.
    """
    cols = np.asarray(cols)
    kc, vc, ukc, uvc = k[cols], v[cols], uk[cols], uv[cols]
    S = scores(q, kc, tau, causal, k_idx=cols)
    P = probabilities(S, L)
    dP = dP_of(do, vc)
    dS = dS_of(P, dP, D)
    F = F_of(q, kc, uq, ukc, tau)
    h = F - alpha[:, None]
    C = C_of(do, uvc)
    Pt = Ptilde_of(C, F, dP, D, alpha)
    St = Stilde_of(P, Pt, E)
    return dict(
        Kt=tau * (St.T @ q + dS.T @ uq),
        Vt=(P * h).T @ do,
        dK=tau * (dS.T @ q),
        dV=P.T @ do,
    )
