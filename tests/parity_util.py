"""Helpers shared by the GPU parity tests (test-side only)."""
import sys

import numpy as np
import torch

import oracle
from workloads import NAMES, as_f64

# Normwise relative error bars: ||x - y||_F / ||y||_F per output tensor.
TOL = {"f32": 1e-4, "bf16": 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def lib():
    import paper_2609_24089_amd as fb
    fb.load_library()
    return fb


def to_dev(x):
    return {k: v.cuda() for k, v in x.items()}


def nrel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def oracle_full(x, scale, causal=False):
    args = [as_f64(x[n]) for n in NAMES]
    return oracle.bob(*args, scale, causal=causal)


def run_gpu_path(xd, scale, use_dq=True, causal=False):
    fb = lib()
    out = fb.bob(*[xd[n] for n in NAMES], scale, causal=causal, use_dq=use_dq)
    torch.cuda.synchronize()
    return out


def global_identities(x, out):
    """I1, I2, I3 (scalar identities) and I5, I6 (zero column sums) evaluated
    on device tensors in float64.  Returns {name: (lhs, rhs, scale)} for the
    scalar identities, where `scale` is the size an inner product of
    unrelated tensors of these norms would have (sum of norm products over
    sqrt(numel)); and {name: max over heads of ||sum_j X_j|| / ||X||_F} for
    the column sums.

    The identities hold exactly for the BoB of attention: Phi is linear in dO
    (I1); dQ, dK are linear in V and dV does not depend on V (I2); S is
    unchanged by Q -> cQ, K -> K/c (I3); P and dS are unchanged by adding a
    constant row to K or to V (I5, I6)."""
    import math
    ip = lambda a, b: float((a.double() * b.double()).sum())
    nrm = lambda a: float(a.double().norm())
    M = x["Q"].numel()
    sq = math.sqrt(M)
    dQUQ, dKUK, dVUV = ip(out["dQ"], x["UQ"]), ip(out["dK"], x["UK"]), ip(out["dV"], x["UV"])
    sQ, sK, sV = nrm(out["dQ"]) * nrm(x["UQ"]), nrm(out["dK"]) * nrm(x["UK"]), nrm(out["dV"]) * nrm(x["UV"])
    scal = {
        "I1": (ip(x["dO"], out["dOt"]), dQUQ + dKUK + dVUV, (nrm(x["dO"]) * nrm(out["dOt"]) + sQ + sK + sV) / sq),
        "I2": (ip(x["V"], out["Vt"]), dQUQ + dKUK, (nrm(x["V"]) * nrm(out["Vt"]) + sQ + sK) / sq),
        "I3": (ip(x["Q"], out["Qt"]) - ip(x["K"], out["Kt"]), dKUK - dQUQ,
               (nrm(x["Q"]) * nrm(out["Qt"]) + nrm(x["K"]) * nrm(out["Kt"]) + sQ + sK) / sq),
    }
    colsum = {}
    for name in ("Kt", "Vt"):
        t = out[name].double().flatten(0, 1)                 # [B*H, N, d]
        colsum[name] = float((t.sum(1).norm(dim=-1) / t.norm(dim=(1, 2))).max())
    return scal, colsum


ROW_KEYS = ("Qt", "dOt", "alpha", "E", "O", "L", "D", "dQ")
SCALAR_TOL = 5e-3     # |lhs - rhs| / scale for I1-I3
COLSUM_TOL = 1e-2     # ||sum_j X_j|| / ||X||_F for I5, I6


def check_rows(x, out, w, rows_per_head, seed, slab=64, causal=False, keys=ROW_KEYS):
    """Row-owned outputs of the GPU path on `rows_per_head` sampled query rows
    of every head against the oracle's `bob_rows` on the same rows (under the
    causal mask row 0, which sees a single key, is always included)."""
    rng = np.random.default_rng(seed)
    got = {k: [] for k in keys}
    want = {k: [] for k in keys}
    for b in range(w.B):
        for h in range(w.H):
            mats = [as_f64(x[n][b, h]) for n in NAMES]
            rows = rng.choice(w.N, size=rows_per_head, replace=False)
            if causal:
                rows[0] = 0
            rows = np.unique(rows)
            for r0 in range(0, len(rows), slab):
                sel = rows[r0:r0 + slab]
                ref = oracle.bob_rows(*mats, w.scale, sel, causal=causal)
                idx = torch.as_tensor(sel, device=out["Qt"].device)
                for k in keys:
                    got[k].append(as_f64(out[k][b, h].index_select(0, idx)))
                    want[k].append(ref[k])
    errs = {k: nrel(np.concatenate(got[k]), np.concatenate(want[k])) for k in keys}
    say("   sampled-row errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL["bf16"], (k, e)


def oracle_workers():
    """Threads for the oracle's slabbed row scalars: the host's cores, at most 16."""
    import os
    return max(1, min(16, os.cpu_count() or 1))


def check_cols(x, out, w, heads, ncols, seed, scalars, causal=False):
    """Column-owned outputs (Kt, Vt, dK, dV) of the GPU path on `ncols`
    sampled key rows of each head in `heads` against the oracle's bob_cols.

    A key row sums over every query row, so bob_cols needs L, D, alpha, E of
    all N rows.  scalars="oracle": the oracle computes them itself for every
    row (row_scalars), so the check is independent of the GPU.
    scalars="gpu": the GPU's own L, D, alpha, E are used (a conditional
    check, for sizes where the oracle cannot form all rows; the caller checks
    those scalars at sampled rows with check_rows).  Multi-head only."""
    import time
    rng = np.random.default_rng(seed)
    got = {k: [] for k in ("Kt", "Vt", "dK", "dV")}
    want = {k: [] for k in got}
    for h in heads:
        mats = [as_f64(x[n][0, h]) for n in NAMES]
        t = time.time()
        if scalars == "oracle":
            step = max(1, w.N // 8)
            report = lambda k, n: k % step < 256 and say(f"   head {h}: oracle row scalars {k}/{n} rows")
            rs = oracle.row_scalars(*mats, w.scale, slab=256, causal=causal, workers=oracle_workers(),
                                    progress=report)
        else:
            rs = {k: as_f64(out[k][0, h]) for k in ("alpha", "E", "L", "D")}
        cols = np.sort(rng.choice(w.N, size=ncols, replace=False))
        ref = oracle.bob_cols(*mats, w.scale, cols, rs["alpha"], rs["E"], rs["L"], rs["D"], causal=causal)
        idx = torch.as_tensor(cols, device=out["Kt"].device)
        for k in got:
            got[k].append(as_f64(out[k][0, h].index_select(0, idx)))
            want[k].append(ref[k])
        say(f"   head {h}: {ncols} key rows, {scalars} row scalars ({time.time() - t:.1f} s)")
    errs = {k: nrel(np.concatenate(got[k]), np.concatenate(want[k])) for k in got}
    say(f"   sampled-column errs ({scalars} row scalars)", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL["bf16"], (k, e)
    return errs


def check_identities(x, out):
    scal, colsum = global_identities(x, out)
    say("   identities", {k: f"{(a - b) / s:.2e}" for k, (a, b, s) in scal.items()},
        {k: f"{v:.2e}" for k, v in colsum.items()})
    for k, (a, b, s) in scal.items():
        assert abs(a - b) <= SCALAR_TOL * s, k
    for k, v in colsum.items():
        assert v <= COLSUM_TOL, k
