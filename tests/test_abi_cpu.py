"""C-ABI checks that need no GPU: the library loads, exports every symbol
include/flashbob.h declares, and rejects bad arguments with the documented
status codes before any HIP call is made (so nothing here touches a device)."""
import ctypes
import os
import re

import pytest

import paper_2609_24089_amd as fb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flashbob.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fb.LIB_PATH):
        from paper_2609_24089_amd.build import build_library
        build_library()
    return fb.load_library()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("attn_fwd_lse", "attn_bwd", "attn_bob_pass1_rows", "attn_bob_pass2_cols",
              "attn_bob3_alpha_rows", "attn_bob3_rows", "bob_supported", "bob_status_string", "bob_version"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_supported_and_strings(lib):
    for d in (32, 64, 128, 256):
        assert lib.bob_supported(fb.BOB_BF16, d) == 1, d
    for d in (32, 64, 128):
        assert lib.bob_supported(fb.BOB_F32, d) == 1, d
    assert lib.bob_supported(fb.BOB_F32, 256) == 0
    assert lib.bob_supported(fb.BOB_BF16, 96) == 0 and lib.bob_supported(7, 64) == 0
    for rc in range(5):
        assert lib.bob_status_string(rc).decode().startswith("BOB_")
    assert lib.bob_status_string(99).decode() == "unknown bob_status"
    assert lib.bob_version().decode().startswith("flashbob")


ALIGNED = 1 << 20          # fake, 16-byte aligned addresses: never dereferenced
MISALIGNED = (1 << 20) + 8


def call(lib, fn, dtype=fb.BOB_BF16, B=1, H=1, N=16, d=64, scale=0.125, ptr=ALIGNED, bad_index=None, causal=0):
    nptr = {"attn_fwd_lse": 5, "attn_bwd": 10, "attn_bob_pass1_rows": 15, "attn_bob_pass2_cols": 13,
            "attn_bob3_alpha_rows": 6, "attn_bob3_rows": 13}[fn]
    ptrs = [ctypes.c_void_p(ptr) for _ in range(nptr)]
    if bad_index is not None:
        ptrs[bad_index] = ctypes.c_void_p(0)
    return getattr(lib, fn)(dtype, B, H, N, d, ctypes.c_float(scale), causal, *ptrs, None)


FNS = ["attn_fwd_lse", "attn_bwd", "attn_bob_pass1_rows", "attn_bob_pass2_cols", "attn_bob3_alpha_rows",
       "attn_bob3_rows"]


@pytest.mark.parametrize("fn", FNS)
def test_rejects_bad_arguments_without_launching(lib, fn):
    assert call(lib, fn, N=-1) == fb.BOB_EINVAL
    assert call(lib, fn, B=-2) == fb.BOB_EINVAL
    assert call(lib, fn, H=-1) == fb.BOB_EINVAL
    assert call(lib, fn, d=0) == fb.BOB_EINVAL
    assert call(lib, fn, scale=float("nan")) == fb.BOB_EINVAL
    assert call(lib, fn, scale=float("inf")) == fb.BOB_EINVAL
    assert call(lib, fn, dtype=5) == fb.BOB_EINVAL
    assert call(lib, fn, d=96) == fb.BOB_EUNSUPPORTED
    assert call(lib, fn, d=16) == fb.BOB_EUNSUPPORTED
    assert call(lib, fn, dtype=fb.BOB_F32, d=256) == fb.BOB_EUNSUPPORTED
    assert call(lib, fn, ptr=MISALIGNED) == fb.BOB_EINVAL
    assert call(lib, fn, ptr=0) == fb.BOB_EINVAL
    assert call(lib, fn, N=(1 << 30) + 1) == fb.BOB_EINVAL
    assert call(lib, fn, B=1 << 20, H=1 << 20) == fb.BOB_EINVAL
    # heads x 32-row tiles past the int range (the column kernels' loop count)
    assert call(lib, fn, H=1 << 10, N=1 << 26) == fb.BOB_EINVAL
    assert call(lib, fn, causal=2) == fb.BOB_EINVAL
    assert call(lib, fn, causal=-1) == fb.BOB_EINVAL


@pytest.mark.parametrize("fn", FNS)
def test_every_pointer_is_checked(lib, fn):
    nptr = {"attn_fwd_lse": 5, "attn_bwd": 10, "attn_bob_pass1_rows": 15, "attn_bob_pass2_cols": 13,
            "attn_bob3_alpha_rows": 6, "attn_bob3_rows": 13}[fn]
    optional = {"attn_bob_pass1_rows": {10}}.get(fn, set())   # dQ may be NULL
    for i in range(nptr):
        if i not in optional:
            assert call(lib, fn, bad_index=i) == fb.BOB_EINVAL, i


def test_optional_dq_pointer(lib):
    # NULL dQ selects the six-accumulator form; a misaligned dQ is rejected
    assert call(lib, "attn_bob_pass1_rows", N=0, ptr=0) == fb.BOB_OK
    ptrs = [ctypes.c_void_p(ALIGNED) for _ in range(15)]
    ptrs[10] = ctypes.c_void_p(MISALIGNED)
    assert lib.attn_bob_pass1_rows(fb.BOB_BF16, 1, 1, 16, 64, ctypes.c_float(0.125), 0, *ptrs, None) == fb.BOB_EINVAL


@pytest.mark.parametrize("fn", FNS)
def test_empty_problem_is_a_no_op(lib, fn):
    # B*H*N == 0 touches no memory, so NULL pointers are fine
    assert call(lib, fn, N=0, ptr=0) == fb.BOB_OK
    assert call(lib, fn, B=0, ptr=0) == fb.BOB_OK
    assert call(lib, fn, H=0, d=128, ptr=0) == fb.BOB_OK
    # an unsupported head dim is reported even for an empty problem
    assert call(lib, fn, N=0, d=80, ptr=0) == fb.BOB_EUNSUPPORTED
    assert call(lib, fn, N=0, ptr=0, causal=1) == fb.BOB_OK


def test_binding_rejects_cpu_tensors():
    import torch
    x = torch.zeros(1, 1, 4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        fb.attn_fwd_lse(x, x, x, 0.125)
    with pytest.raises(TypeError):
        fb._dtype_code(torch.zeros(1, dtype=torch.float16))


def test_attention_wrapper_rejects_host_tensors():
    """The differentiable wrapper has no host path: CPU tensors are refused
    before any library call."""
    import torch
    x = torch.zeros(1, 1, 8, 64)
    with pytest.raises(ValueError, match="ROCm device"):
        fb.attention(x, x, x)


GQA_NPTR = {"attn_fwd_lse_gqa": 5, "attn_bwd_gqa": 10, "attn_bob_pass1_rows_gqa": 15, "attn_bob_pass2_cols_gqa": 13}


def call_gqa(lib, fn, H=4, Hkv=2, dtype=fb.BOB_BF16, B=1, N=16, d=64, scale=0.125, ptr=ALIGNED, bad_index=None,
             causal=0):
    ptrs = [ctypes.c_void_p(ptr) for _ in range(GQA_NPTR[fn])]
    if bad_index is not None:
        ptrs[bad_index] = ctypes.c_void_p(0)
    return getattr(lib, fn)(dtype, B, H, Hkv, N, d, ctypes.c_float(scale), causal, *ptrs, None)


def test_header_declares_the_grouped_entry_points():
    names = declared_functions()
    for n in GQA_NPTR:
        assert n in names


@pytest.mark.parametrize("fn", sorted(GQA_NPTR))
def test_grouped_heads_are_validated(lib, fn):
    assert call_gqa(lib, fn, H=4, Hkv=0) == fb.BOB_EINVAL
    assert call_gqa(lib, fn, H=4, Hkv=-1) == fb.BOB_EINVAL
    assert call_gqa(lib, fn, H=4, Hkv=3) == fb.BOB_EINVAL       # 4 is not a multiple of 3
    assert call_gqa(lib, fn, H=4, Hkv=8) == fb.BOB_EINVAL       # more key/value heads than query heads
    assert call_gqa(lib, fn, d=96) == fb.BOB_EUNSUPPORTED
    assert call_gqa(lib, fn, scale=float("nan")) == fb.BOB_EINVAL
    assert call_gqa(lib, fn, causal=2) == fb.BOB_EINVAL
    assert call_gqa(lib, fn, ptr=MISALIGNED) == fb.BOB_EINVAL
    # empty problems touch no memory
    assert call_gqa(lib, fn, N=0, ptr=0) == fb.BOB_OK
    assert call_gqa(lib, fn, H=0, Hkv=0, ptr=0) == fb.BOB_OK


@pytest.mark.parametrize("fn", sorted(GQA_NPTR))
def test_grouped_entry_points_check_every_pointer(lib, fn):
    optional = {"attn_bob_pass1_rows_gqa": {10}}.get(fn, set())   # dQ may be NULL
    for i in range(GQA_NPTR[fn]):
        if i not in optional:
            assert call_gqa(lib, fn, bad_index=i) == fb.BOB_EINVAL, i


def test_binding_checks_group_shapes():
    import torch
    q = torch.zeros(1, 4, 8, 64, dtype=torch.bfloat16)
    k3 = torch.zeros(1, 3, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="multiple of the key/value heads"):
        fb.attn_fwd_lse(q, k3, k3, 0.125)
    k2 = torch.zeros(1, 2, 9, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="must match the query side"):
        fb.attn_fwd_lse(q, k2, k2, 0.125)


def opts(parts=0, wave_sets=0, flush_tiles=0):
    return ctypes.byref(fb.ColumnOpts(parts, wave_sets, flush_tiles))


def call_ws(lib, ws=ALIGNED, nbytes=1 << 40, bad_index=None, dtype=fb.BOB_BF16, B=1, H=4, Hkv=1, N=1000, d=64,
            causal=1, o=None):
    ptrs = [ctypes.c_void_p(ALIGNED) for _ in range(13)]
    if bad_index is not None:
        ptrs[bad_index] = ctypes.c_void_p(0)
    return lib.attn_bob_pass2_cols_gqa_ws(dtype, B, H, Hkv, N, d, ctypes.c_float(0.125), causal, *ptrs,
                                          opts(4) if o is None else o, ctypes.c_void_p(ws), nbytes, None)


def call_bwd_ws(lib, ws=ALIGNED, nbytes=1 << 40, bad_index=None, dtype=fb.BOB_BF16, B=1, H=4, Hkv=1, N=1000,
                d=64, causal=1, o=None):
    ptrs = [ctypes.c_void_p(ALIGNED) for _ in range(10)]
    if bad_index is not None:
        ptrs[bad_index] = ctypes.c_void_p(0)
    return lib.attn_bwd_gqa_ws(dtype, B, H, Hkv, N, d, ctypes.c_float(0.125), causal, *ptrs,
                               opts(4) if o is None else o, ctypes.c_void_p(ws), nbytes, None)


def test_column_split_workspace(lib):
    """With a forced part count the workspace is parts x {Kt, Vt} x B*Hkv*N*d
    fp32 values, and the split calls reject a missing, misaligned or short
    workspace (and every bad tensor pointer) before any launch."""
    need = 4 * 2 * 1 * 1 * 1000 * 64 * 4
    assert lib.bob_pass2_workspace_bytes(fb.BOB_BF16, 1, 4, 1, 1000, 64, 1, opts(4)) == need
    assert lib.bob_pass2_workspace_bytes(fb.BOB_F32, 2, 4, 2, 100, 32, 0, opts(4)) == 4 * 2 * 2 * 2 * 100 * 32 * 4
    # empty, invalid and unsupported problems need none (the call reports them)
    assert lib.bob_pass2_workspace_bytes(fb.BOB_BF16, 1, 4, 1, 0, 64, 1, opts(4)) == 0
    assert lib.bob_pass2_workspace_bytes(fb.BOB_BF16, 1, 4, 3, 1000, 64, 1, opts(4)) == 0
    assert lib.bob_pass2_workspace_bytes(fb.BOB_BF16, 1, 4, 1, 1000, 96, 1, opts(4)) == 0
    assert lib.bob_pass2_workspace_bytes(fb.BOB_BF16, 1, 4, 1, 1000, 64, 1, opts(9)) == 0
    assert call_ws(lib, ws=0) == fb.BOB_EINVAL
    assert call_ws(lib, ws=MISALIGNED) == fb.BOB_EINVAL
    assert call_ws(lib, nbytes=need - 1) == fb.BOB_EINVAL
    for i in range(13):
        assert call_ws(lib, bad_index=i) == fb.BOB_EINVAL, i
    assert call_ws(lib, H=4, Hkv=3) == fb.BOB_EINVAL
    assert call_ws(lib, d=96) == fb.BOB_EUNSUPPORTED
    assert call_ws(lib, N=0, ws=0) == fb.BOB_OK               # empty: nothing to do
    # the first backward's split: same size rule and the same checks
    assert lib.bob_bwd_workspace_bytes(fb.BOB_BF16, 1, 4, 1, 1000, 64, 1, opts(4)) == need
    assert lib.bob_bwd_workspace_bytes(fb.BOB_BF16, 1, 4, 1, 1000, 96, 1, opts(4)) == 0
    assert call_bwd_ws(lib, ws=0) == fb.BOB_EINVAL
    assert call_bwd_ws(lib, ws=MISALIGNED) == fb.BOB_EINVAL
    assert call_bwd_ws(lib, nbytes=need - 1) == fb.BOB_EINVAL
    for i in range(10):
        assert call_bwd_ws(lib, bad_index=i) == fb.BOB_EINVAL, i
    assert call_bwd_ws(lib, N=0, ws=0) == fb.BOB_OK
    # unsplit: no workspace needed, none checked
    assert lib.bob_pass2_workspace_bytes(fb.BOB_BF16, 1, 4, 1, 1000, 64, 1, opts(1)) == 0
    assert lib.bob_bwd_workspace_bytes(fb.BOB_BF16, 1, 4, 1, 1000, 64, 1, opts(1)) == 0


def test_column_opts_are_validated(lib):
    """Requests out of range are BOB_EINVAL in the calls and the queries;
    sections where no sectioned form is built are BOB_EUNSUPPORTED."""
    for bad in (opts(-1), opts(9), opts(0, -1), opts(0, 3), opts(0, 0, -2)):
        assert call_ws(lib, o=bad) == fb.BOB_EINVAL
        assert call_bwd_ws(lib, o=bad) == fb.BOB_EINVAL
        for kernel in (fb.BOB_COLUMNS_BWD, fb.BOB_COLUMNS_PASS2):
            assert lib.bob_column_layout(kernel, fb.BOB_BF16, 1, 4, 1, 1000, 64, 1, bad, None, None) == fb.BOB_EINVAL
    assert lib.bob_column_layout(7, fb.BOB_BF16, 1, 4, 1, 1000, 64, 1, None, None, None) == fb.BOB_EINVAL
    for dt, d in ((fb.BOB_BF16, 256), (fb.BOB_F32, 64)):
        assert call_ws(lib, dtype=dt, d=d, o=opts(1, 1, 8)) == fb.BOB_EUNSUPPORTED
        assert call_bwd_ws(lib, dtype=dt, d=d, o=opts(1, 1, 8)) == fb.BOB_EUNSUPPORTED
        # automatic sections there fall back to one section
        assert lib.bob_column_layout(fb.BOB_COLUMNS_PASS2, dt, 1, 1, 1, 1 << 20, d, 0, opts(1), None, None) == 0


def layout(lib, kernel, o, dtype=fb.BOB_BF16, B=1, H=4, Hkv=1, N=1000, d=64, causal=1):
    got = fb.ColumnOpts()
    nbytes = ctypes.c_int64(-1)
    rc = lib.bob_column_layout(kernel, dtype, B, H, Hkv, N, d, causal, o, ctypes.byref(got), ctypes.byref(nbytes))
    assert rc == fb.BOB_OK
    return (got.parts, got.wave_sets, got.flush_tiles), nbytes.value


def test_column_layout_resolves_requests(lib):
    """Forced requests come back as given; a split runs one wave set; a long
    stream gets sections of 1024 tiles when sections are automatic (bf16
    d <= 128), and asking for one section (-1) keeps a single chain."""
    for kernel in (fb.BOB_COLUMNS_BWD, fb.BOB_COLUMNS_PASS2):
        assert layout(lib, kernel, opts(3, 2, 5)) == ((3, 1, 5), 3 * 2 * 1000 * 64 * 4)
        assert layout(lib, kernel, opts(1, 1, 2)) == ((1, 1, 2), 0)
        assert layout(lib, kernel, opts(1, 2, -1)) == ((1, 2, -1), 0)
        # B1 H1 N = 2^20, d = 64: 32768 streamed tiles in one chain -> sections
        for d in (32, 64, 128):
            assert layout(lib, kernel, opts(1, 1), H=1, N=1 << 20, d=d, causal=0) == ((1, 1, 1024), 0)
            assert layout(lib, kernel, opts(1, 1, -1), H=1, N=1 << 20, d=d, causal=0) == ((1, 1, -1), 0)
            # 16384 tiles stay in one chain; split in 8 parts the chain is short again
            assert layout(lib, kernel, opts(1, 1), H=1, N=1 << 19, d=d, causal=0) == ((1, 1, -1), 0)
            assert layout(lib, kernel, opts(8, 1), H=1, N=1 << 20, d=d, causal=0)[0] == (8, 1, -1)
        # grouped heads lengthen the stream: 16 query heads x 2048 tiles
        assert layout(lib, kernel, opts(1, 1), H=16, Hkv=1, N=65536, d=64, causal=0)[0] == (1, 1, 1024)
    # the empty problem has the trivial layout
    assert layout(lib, fb.BOB_COLUMNS_PASS2, None, N=0) == ((1, 1, -1), 0)


def call_noalloc(lib, o=None, bad_index=None, dtype=fb.BOB_BF16, B=1, H=16, Hkv=1, N=16384, d=128, causal=1):
    ptrs = [ctypes.c_void_p(ALIGNED) for _ in range(13)]
    if bad_index is not None:
        ptrs[bad_index] = ctypes.c_void_p(0)
    return lib.attn_bob_pass2_cols_gqa_noalloc(dtype, B, H, Hkv, N, d, ctypes.c_float(0.125), causal, *ptrs, o,
                                               None)


def test_noalloc_rejects_before_launching(lib):
    """The allocation-free Pass 2 checks its problem, request and pointers
    like the *_ws call, and refuses a forced split whose partial sums would
    not fit its static scratch (BOB_ESCRATCH), all before any HIP call."""
    cap = lib.bob_scratch_bytes()
    assert cap == 64 << 20
    # B1 Hkv1 N16384 d128: 16 MiB of fp32 per {Kt, Vt} part pair x parts
    per_part = 2 * 16384 * 128 * 4
    assert 4 * per_part <= cap < 5 * per_part
    assert call_noalloc(lib, opts(5)) == fb.BOB_ESCRATCH
    assert call_noalloc(lib, opts(8)) == fb.BOB_ESCRATCH
    assert lib.bob_status_string(fb.BOB_ESCRATCH).decode().startswith("BOB_ESCRATCH")
    for bad in (opts(-1), opts(0, 3), opts(0, 0, -2)):
        assert call_noalloc(lib, bad) == fb.BOB_EINVAL
    for i in range(13):
        assert call_noalloc(lib, opts(1), bad_index=i) == fb.BOB_EINVAL, i
    assert call_noalloc(lib, opts(1), d=96) == fb.BOB_EUNSUPPORTED
    assert call_noalloc(lib, opts(1), H=4, Hkv=3) == fb.BOB_EINVAL
    assert call_noalloc(lib, None, N=0) == fb.BOB_OK
