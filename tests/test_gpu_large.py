"""GPU checks at the three large workloads, in the launch configuration the
benchmark times (Pass 1 with dQ, one stream):

* B=1 H=16 N=16384 d=128 (Q, K ~ 0.5 N(0,1), seed 2): row-owned outputs on
  64 sampled query rows of every head; column-owned outputs (Kt, Vt, dK, dV)
  on 256 sampled key rows of head 0, using row scalars the oracle computes
  for all 16384 rows of that head itself;
* B=1 H=8 N=65536 d=64 (seed 3) and B=1 H=4 N=262144 d=64 (seed 4): row-owned
  outputs on sampled query rows (256 per head at N=262144, i.e. 1024 rows);
  column-owned outputs through identities that hold at any size;
* the identities I1-I3, I5, I6 on the full outputs of every workload;
* footprint: the two BoB passes allocate nothing beyond caller buffers.
Normwise bar on every sampled set: 2e-2 (bf16 inputs, fp32 accumulation)."""
import numpy as np
import pytest
import torch

import oracle
from tests.parity_util import TOL, check_identities, check_rows, lib, nrel, run_gpu_path, say, to_dev
from workloads import NAMES, WORKLOADS, as_f64, workload_inputs

pytestmark = pytest.mark.gpu

def test_n16384_d128():
    w = WORKLOADS["bf16_b1h16_n16384_d128"]
    say(f"[large] {w.name}: GPU path")
    x = workload_inputs(w)
    xd = to_dev(x)
    out = run_gpu_path(xd, w.scale)
    check_rows(x, out, w, rows_per_head=64, seed=1002)
    say("[large] column outputs of head 0 (oracle row scalars for all rows)")
    mats = [as_f64(x[n][0, 0]) for n in NAMES]
    rs = oracle.row_scalars(*mats, w.scale, slab=1024)
    cols = np.sort(np.random.default_rng(2002).choice(w.N, size=256, replace=False))
    ref = oracle.bob_cols(*mats, w.scale, cols, rs["alpha"], rs["E"], rs["L"], rs["D"])
    idx = torch.as_tensor(cols, device=out["Kt"].device)
    errs = {k: nrel(as_f64(out[k][0, 0].index_select(0, idx)), ref[k]) for k in ("Kt", "Vt", "dK", "dV")}
    say("   sampled-column errs", {k: f"{v:.2e}" for k, v in errs.items()})
    for k, e in errs.items():
        assert e <= TOL["bf16"], (k, e)
    check_identities(xd, out)


def test_n65536_d64():
    w = WORKLOADS["bf16_b1h8_n65536_d64"]
    say(f"[large] {w.name}: GPU path")
    x = workload_inputs(w)
    xd = to_dev(x)
    out = run_gpu_path(xd, w.scale)
    check_rows(x, out, w, rows_per_head=48, seed=1003)
    check_identities(xd, out)


def test_n262144_d64_and_footprint():
    w = WORKLOADS["bf16_b1h4_n262144_d64"]
    say(f"[large] {w.name}: GPU path")
    fb = lib()
    x = workload_inputs(w)
    xd = to_dev(x)
    Q, K, V, dO, UQ, UK, UV = (xd[n] for n in NAMES)
    O, L = fb.attn_fwd_lse(Q, K, V, w.scale)
    dQ, dK, dV, D = fb.attn_bwd(Q, K, V, O, dO, L, w.scale)
    outs1 = (torch.empty_like(Q), torch.empty_like(Q),
             torch.empty_like(L), torch.empty_like(L))
    outs2 = (torch.empty_like(Q), torch.empty_like(Q))
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    fb.attn_bob_pass1_rows(Q, K, V, O, dO, UQ, UK, UV, L, D, w.scale, dQ=dQ, out=outs1)
    fb.attn_bob_pass2_cols(Q, K, V, dO, UQ, UK, UV, L, D, outs1[2], outs1[3], w.scale, out=outs2)
    torch.cuda.synchronize()
    # the library allocates nothing: the passes add no device memory
    assert torch.cuda.max_memory_allocated() == before
    extra = outs1[2].nbytes + outs1[3].nbytes      # alpha, E: the only BoB-only state
    assert extra == 2 * 4 * w.B * w.H * w.N
    out = dict(O=O, L=L, D=D, dQ=dQ, dK=dK, dV=dV, Qt=outs1[0], dOt=outs1[1], alpha=outs1[2],
               E=outs1[3], Kt=outs2[0], Vt=outs2[1])
    check_rows(x, out, w, rows_per_head=256, seed=1004)
    check_identities(xd, out)
