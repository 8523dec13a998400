"""GPU checks at the large workloads, in the launch configuration the
benchmark times (Pass 1 with dQ, one stream):

* B=1 H=16 N=16384 d=128 (Q, K ~ 0.5 N(0,1), seed 2): row-owned outputs on
  64 sampled query rows of every head; column-owned outputs (Kt, Vt, dK, dV)
  on 256 sampled key rows of head 0, using row scalars the oracle computes
  for all 16384 rows of that head itself;
* B=1 H=8 N=65536 d=64 (seed 3): row-owned outputs on 256 sampled query rows
  of every head; column-owned outputs on 256 sampled key rows of head 0,
  using row scalars the oracle computes for all 65536 rows of that head, and
  on 64 sampled key rows of every other head given the GPU's row scalars
  (conditional, see below);
* B=1 H=4 N=262144 d=64 (seed 4): row-owned outputs on 256 sampled query
  rows per head (1024 rows); column-owned outputs on 256 sampled key rows of
  head 0, using row scalars the oracle computes for all 262144 rows of that
  head (about two minutes of host time), and on 256 sampled key rows of every
  head given the GPU's L, D, alpha, E.  The latter is a conditional check: a
  key row sums over all 262144 query rows, so it checks the column
  arithmetic given the row scalars, which are checked separately at the
  sampled query rows;
* B=1 H=16 N=8192 d=256 (seed 15; Pass 1 in one workgroup per row block,
  Pass 2 in wave pairs): row-owned outputs on 32 sampled query rows of every
  head; column-owned outputs on 128 sampled key rows of head 0, using row
  scalars the oracle computes for all 8192 rows of that head;
* the identities I1-I3, I5, I6 on the full outputs of every workload;
* footprint: the two BoB passes allocate nothing beyond caller buffers.
Normwise bar on every sampled set: 2e-2 (bf16 inputs, fp32 accumulation)."""
import pytest
import torch

from tests.parity_util import check_cols, check_identities, check_rows, lib, run_gpu_path, say, to_dev
from workloads import NAMES, WORKLOADS, workload_inputs

pytestmark = pytest.mark.gpu

def test_n16384_d128():
    w = WORKLOADS["bf16_b1h16_n16384_d128"]
    say(f"[large] {w.name}: GPU path")
    x = workload_inputs(w)
    xd = to_dev(x)
    out = run_gpu_path(xd, w.scale)
    check_rows(x, out, w, rows_per_head=64, seed=1002)
    say("[large] column outputs of head 0 (oracle row scalars for all rows)")
    check_cols(x, out, w, heads=[0], ncols=256, seed=2002, scalars="oracle")
    check_identities(xd, out)


def test_n8192_d256():
    w = WORKLOADS["bf16_b1h16_n8192_d256"]
    say(f"[large] {w.name}: GPU path")
    x = workload_inputs(w)
    xd = to_dev(x)
    out = run_gpu_path(xd, w.scale)
    check_rows(x, out, w, rows_per_head=32, seed=1005)
    say("[large] column outputs of head 0 (oracle row scalars for all rows)")
    check_cols(x, out, w, heads=[0], ncols=128, seed=2005, scalars="oracle")
    check_identities(xd, out)


def test_n65536_d64():
    w = WORKLOADS["bf16_b1h8_n65536_d64"]
    say(f"[large] {w.name}: GPU path")
    x = workload_inputs(w)
    xd = to_dev(x)
    out = run_gpu_path(xd, w.scale)
    check_rows(x, out, w, rows_per_head=256, seed=1003)
    say("[large] column outputs of head 0 (oracle row scalars for all rows)")
    check_cols(x, out, w, heads=[0], ncols=256, seed=2003, scalars="oracle")
    say("[large] column outputs of heads 1-7 (GPU row scalars)")
    check_cols(x, out, w, heads=range(1, w.H), ncols=64, seed=2013, scalars="gpu")
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
    say("[large] column outputs of head 0 (oracle row scalars for all rows)")
    check_cols(x, out, w, heads=[0], ncols=256, seed=2014, scalars="oracle")
    say("[large] column outputs, 256 key rows per head (GPU row scalars, checked above at the sampled rows)")
    check_cols(x, out, w, heads=range(w.H), ncols=256, seed=2004, scalars="gpu")
    check_identities(xd, out)
