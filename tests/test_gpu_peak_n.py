"""GPU checks in the long-sequence regime of one MI355X (B=H=1, d=64, bf16,
dense, seed 7: the inputs the benchmark's peak-N sweep draws), in the launch
configuration the benchmark times, at N = 2^19 ... 2^22:

* row-owned outputs on sampled query rows against the oracle;
* column-owned outputs (Kt, Vt, dK, dV) on sampled key rows against the
  oracle's column slice, given the row scalars (L, D, alpha, E) the GPU
  produced, which are themselves checked at the sampled rows (a conditional
  check: the oracle cannot form alpha, E for millions of rows in test time);
* the scalar identities I1-I3 and the zero column sums I5 (sum_j Kt_j = 0),
  I6 (sum_j Vt_j = 0) and sum_j dK_j = 0 on the full outputs at every N.

The column sums are what a one-signed rounding error in a long accumulation
shows: every column adds it, so the sum over N columns grows like N while
the norm it is compared with grows like sqrt(N).  Above 16384 streamed tiles
per accumulator chain the column kernels accumulate in sections of 1024
tiles (bob_column_opts.flush_tiles, automatic), which keeps these sums at the
bf16 rounding floor; the test checks that the automatic layout does so."""
import numpy as np
import pytest
import torch

from tests.parity_util import (COLSUM_TOL, SCALAR_TOL, check_cols, check_rows, global_identities, lib, say,
                               to_dev)
from workloads import Workload, workload_inputs

pytestmark = pytest.mark.gpu


def dk_colsum(dK):
    t = dK.double().flatten(0, 1)
    return float((t.sum(1).norm(dim=-1) / t.norm(dim=(1, 2))).max())


@pytest.mark.parametrize("logn", [19, 20, 21, 22])
def test_long_sequence(logn):
    fb = lib()
    N = 1 << logn
    w = Workload(f"bf16_b1h1_n{N}_d64", 1, 1, N, 64, "bf16", 7)
    for kernel, name in ((fb.BOB_COLUMNS_BWD, "bwd"), (fb.BOB_COLUMNS_PASS2, "pass2")):
        got, _ = fb.column_layout(kernel, torch.bfloat16, 1, 1, 1, N, 64, False)
        say(f"[peak-n] N={N} {name} column layout {got}")
        # more than 16384 streamed tiles per chain -> sections of 1024
        assert got.flush_tiles == (1024 if N // 32 > 16384 * got.parts * got.wave_sets else -1)
    say(f"[peak-n] {w.name}: generating inputs")
    x = workload_inputs(w)
    xd = to_dev(x)
    say(f"[peak-n] {w.name}: GPU path")
    out = fb.bob(*[xd[n] for n in ("Q", "K", "V", "dO", "UQ", "UK", "UV")], w.scale)
    torch.cuda.synchronize()
    say(f"[peak-n] {w.name}: oracle rows and columns")
    check_rows(x, out, w, rows_per_head=24, seed=7007, slab=8)
    check_cols(x, out, w, heads=[0], ncols=32, seed=7008, scalars="gpu")
    scal, colsum = global_identities(xd, out)
    colsum["dK"] = dk_colsum(out["dK"])
    say("   identities", {k: f"{(a - b) / s:.2e}" for k, (a, b, s) in scal.items()},
        {k: f"{v:.2e}" for k, v in colsum.items()})
    for k, (a, b, s) in scal.items():
        assert abs(a - b) <= SCALAR_TOL * s, k
    for k, v in colsum.items():
        assert v <= COLSUM_TOL, (k, v)
