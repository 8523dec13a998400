"""GPU check of attn_bob_pass2_cols_gqa_noalloc, the Pass 2 entry point for
callers that cannot allocate: its split layout keeps the fp32 partial sums in
the library's static scratch buffer instead of a caller's workspace.  Its
Kt, Vt must equal attn_bob_pass2_cols_gqa_ws's with the same resolved layout
bit for bit, over two calls in a row with the second on a smaller problem
(the scratch keeps the first call's contents, which a split never reads);
with automatic parts on a problem whose automatic split would overflow the
scratch, the call takes the largest part count that fits; the calls
themselves allocate no device memory."""
import numpy as np
import pytest
import torch

from tests.parity_util import say
from workloads import NAMES, make_gqa_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture
def fb():
    import paper_2609_24089_amd as m
    m.load_library()
    return m


def prepared(fb, B, H, Hkv, N, d, causal, seed):
    x = {k: v.cuda() for k, v in make_gqa_inputs(B, H, Hkv, N, d, "bf16", seed).items()}
    Q, K, V, dO, UQ, UK, UV = (x[n] for n in NAMES)
    scale = 1.0 / np.sqrt(d)
    O, L = fb.attn_fwd_lse(Q, K, V, scale, causal)
    dQ, dK, dV, D = fb.attn_bwd(Q, K, V, O, dO, L, scale, causal)
    Qt, dOt, al, E = fb.attn_bob_pass1_rows(Q, K, V, O, dO, UQ, UK, UV, L, D, scale, causal, dQ=dQ)
    torch.cuda.synchronize()
    return (Q, K, V, dO, UQ, UK, UV, L, D, al, E), scale


def both(fb, args, scale, causal, cols_ws, cols_noalloc):
    """Kt, Vt from the *_ws call and from the allocation-free call (into
    preallocated outputs, so the latter allocates nothing at all)."""
    ref = fb.attn_bob_pass2_cols(*args, scale, causal, columns=cols_ws)
    K = args[1]
    out = (torch.empty_like(K), torch.empty_like(K))
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    got = fb.attn_bob_pass2_cols_noalloc(*args, scale, causal, out=out, columns=cols_noalloc)
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated() == before
    return ref, got


@pytest.mark.parametrize("causal", [True, False])
def test_noalloc_matches_ws_on_two_calls(fb, causal):
    lib = fb.load_library()
    cases = [(1, 16, 1, 2048, 128, 4, 190), (1, 8, 2, 1000, 64, 3, 191)]   # the second is smaller
    for B, H, Hkv, N, d, parts, seed in cases:
        args, scale = prepared(fb, B, H, Hkv, N, d, causal, seed)
        cols = fb.ColumnOpts(parts, 0, 0)
        lay, nbytes = fb.column_layout(fb.BOB_COLUMNS_PASS2, torch.bfloat16, B, H, Hkv, N, d, causal, cols)
        assert lay.parts == parts and 0 < nbytes <= lib.bob_scratch_bytes()
        ref, got = both(fb, args, scale, causal, cols, cols)
        say(f"[noalloc] B{B} H{H} Hkv{Hkv} N{N} d{d} causal={causal} parts {parts}: "
            f"max |diff| Kt {float((ref[0].float() - got[0].float()).abs().max()):.1e}")
        assert torch.equal(ref[0], got[0]) and torch.equal(ref[1], got[1])


def test_noalloc_caps_automatic_parts(fb):
    """Causal multi-query B1 H16 N16384 d128: the automatic split would use 8
    parts (128 MiB of partial sums); the allocation-free call fits 4 into its
    64 MiB and equals the *_ws call forced to 4 parts."""
    lib = fb.load_library()
    B, H, Hkv, N, d = 1, 16, 1, 16384, 128
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    auto, nbytes = fb.column_layout(fb.BOB_COLUMNS_PASS2, torch.bfloat16, B, H, Hkv, N, d, True)
    per_part = 2 * B * Hkv * N * d * 4
    fit = min(8, lib.bob_scratch_bytes() // per_part)
    say(f"[noalloc] automatic parts {auto.parts} ({nbytes >> 20} MiB) on {cus} CUs; scratch fits {fit}")
    args, scale = prepared(fb, B, H, Hkv, N, d, True, 192)
    want = fb.ColumnOpts(min(auto.parts, fit) if min(auto.parts, fit) >= 2 else 1, 0, 0)
    ref, got = both(fb, args, scale, True, want, None)
    assert torch.equal(ref[0], got[0]) and torch.equal(ref[1], got[1])
    # a forced split that does not fit is refused
    if 8 * per_part > lib.bob_scratch_bytes():
        with pytest.raises(RuntimeError, match="BOB_ESCRATCH"):
            fb.attn_bob_pass2_cols_noalloc(*args, scale, True, columns=fb.ColumnOpts(8, 0, 0))
