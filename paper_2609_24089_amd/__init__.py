"""Exact attention backward-over-backward (FlashBoB) on MI355X.

Thin Python binding over libflashbob.so (include/flashbob.h).  The entry
points keep the C names (the grouped-query variants are chosen from the
tensor shapes); each one only checks and marshals torch-ROCm tensors
(device memory and the current stream) and calls the library, so every step
of the computation runs in the gfx950 kernels.  There is no fallback: if the
library is missing, importing the binding raises.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libflashbob.so")

BOB_F32 = 0
BOB_BF16 = 1
BOB_OK, BOB_EINVAL, BOB_EUNSUPPORTED, BOB_ELAUNCH, BOB_ESCRATCH = 0, 1, 2, 3, 4
BOB_COLUMNS_BWD, BOB_COLUMNS_PASS2 = 0, 1

_lib = None


class ColumnOpts(ctypes.Structure):
    """bob_column_opts: layout requests for the column kernels (the first
    backward's dK, dV and Pass 2's Kt, Vt); 0 = automatic in every field.
    parts: workgroups per column block (1..8); wave_sets: 1 or 2;
    flush_tiles: streamed tiles per accumulation section (>= 1, or -1 for
    one section).  See include/flashbob.h."""
    _fields_ = [("parts", ctypes.c_int32), ("wave_sets", ctypes.c_int32), ("flush_tiles", ctypes.c_int32)]

    def __repr__(self):
        return f"ColumnOpts(parts={self.parts}, wave_sets={self.wave_sets}, flush_tiles={self.flush_tiles})"


def load_library():
    """Load libflashbob.so (built by paper_2609_24089_amd.build); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2609_24089_amd.build` "
            "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, f32, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
    common = [i32, i64, i64, i64, i64, f32, i32]
    lib.attn_fwd_lse.argtypes = common + [vp] * 5 + [vp]
    lib.attn_bwd.argtypes = common + [vp] * 10 + [vp]
    lib.attn_bob_pass1_rows.argtypes = common + [vp] * 15 + [vp]
    lib.attn_bob_pass2_cols.argtypes = common + [vp] * 13 + [vp]
    lib.attn_bob3_alpha_rows.argtypes = common + [vp] * 6 + [vp]
    lib.attn_bob3_rows.argtypes = common + [vp] * 13 + [vp]
    common_gqa = [i32, i64, i64, i64, i64, i64, f32, i32]  # ... H, Hkv, N, ...
    lib.attn_fwd_lse_gqa.argtypes = common_gqa + [vp] * 5 + [vp]
    lib.attn_bwd_gqa.argtypes = common_gqa + [vp] * 10 + [vp]
    lib.attn_bob_pass1_rows_gqa.argtypes = common_gqa + [vp] * 15 + [vp]
    lib.attn_bob_pass2_cols_gqa.argtypes = common_gqa + [vp] * 13 + [vp]
    for fn in ("attn_fwd_lse", "attn_bwd", "attn_bob_pass1_rows", "attn_bob_pass2_cols",
               "attn_bob3_alpha_rows", "attn_bob3_rows", "attn_fwd_lse_gqa", "attn_bwd_gqa",
               "attn_bob_pass1_rows_gqa", "attn_bob_pass2_cols_gqa"):
        getattr(lib, fn).restype = i32
    lib.bob_supported.argtypes = [i32, i64]
    lib.bob_supported.restype = i32
    lib.bob_status_string.argtypes = [i32]
    lib.bob_status_string.restype = ctypes.c_char_p
    lib.bob_version.argtypes = []
    lib.bob_version.restype = ctypes.c_char_p
    opts_p = ctypes.POINTER(ColumnOpts)
    lib.bob_pass2_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i64, i32, opts_p]
    lib.bob_pass2_workspace_bytes.restype = i64
    lib.bob_bwd_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i64, i32, opts_p]
    lib.bob_bwd_workspace_bytes.restype = i64
    lib.bob_column_layout.argtypes = [i32, i32, i64, i64, i64, i64, i64, i32, opts_p, opts_p,
                                      ctypes.POINTER(i64)]
    lib.bob_column_layout.restype = i32
    lib.attn_bob_pass2_cols_gqa_ws.argtypes = common_gqa + [vp] * 13 + [opts_p, vp, i64] + [vp]
    lib.attn_bob_pass2_cols_gqa_ws.restype = i32
    lib.attn_bwd_gqa_ws.argtypes = common_gqa + [vp] * 10 + [opts_p, vp, i64] + [vp]
    lib.attn_bwd_gqa_ws.restype = i32
    lib.attn_bob_pass2_cols_gqa_noalloc.argtypes = common_gqa + [vp] * 13 + [opts_p] + [vp]
    lib.attn_bob_pass2_cols_gqa_noalloc.restype = i32
    lib.bob_scratch_bytes.argtypes = []
    lib.bob_scratch_bytes.restype = i64
    _lib = lib
    return lib


def status_string(rc):
    return load_library().bob_status_string(int(rc)).decode()


def _opts(columns):
    """A ColumnOpts (or None, all automatic) as the pointer argument of the
    *_ws calls and queries."""
    if columns is None:
        return None
    if not isinstance(columns, ColumnOpts):
        raise TypeError("columns must be a ColumnOpts or None")
    return ctypes.byref(columns)


def column_layout(kernel, dtype, B, H, Hkv, N, d, causal=False, columns=None, device=None):
    """bob_column_layout: the layout the column kernel `kernel`
    (BOB_COLUMNS_BWD or BOB_COLUMNS_PASS2) runs for this problem and request
    on `device` (default: the current device).  Returns (ColumnOpts with the
    resolved parts, wave_sets, flush_tiles (-1: one section), workspace
    bytes)."""
    lib = load_library()
    code = _dtype_code(torch.empty(0, dtype=dtype))
    got = ColumnOpts()
    nbytes = ctypes.c_int64(0)
    with torch.cuda.device(device if device is not None else torch.cuda.current_device()):
        rc = lib.bob_column_layout(kernel, code, B, H, Hkv, N, d, int(bool(causal)), _opts(columns),
                                   ctypes.byref(got), ctypes.byref(nbytes))
    if rc != BOB_OK:
        raise RuntimeError(status_string(rc))
    return got, nbytes.value


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return BOB_BF16
    if t.dtype == torch.float32:
        return BOB_F32
    raise TypeError(f"unsupported dtype {t.dtype}; expected torch.bfloat16 or torch.float32")


def _check_mats(*ts):
    ref = ts[0]
    if ref.dim() != 4:
        raise ValueError("matrices must be [B, H, N, d]")
    for t in ts:
        if t.shape != ref.shape or t.dtype != ref.dtype or t.device != ref.device:
            raise ValueError("all matrices must share shape, dtype and device")
        if not t.is_contiguous():
            raise ValueError("matrices must be contiguous")
        if t.device.type != "cuda":
            raise ValueError("matrices must be on a ROCm device")
    return ref.shape


def _check_groups(qside, kside):
    """Query-side matrices [B, H, N, d] and key/value-side matrices
    [B, Hkv, N, d] with H a multiple of Hkv (grouped-query attention; Hkv = H
    is multi-head attention).  Returns (B, H, Hkv, N, d)."""
    q, k = qside[0], kside[0]
    if q.dim() != 4 or k.dim() != 4:
        raise ValueError("matrices must be [B, H, N, d]")
    B, H, N, d = q.shape
    kB, Hkv, kN, kd = k.shape
    if (kB, kN, kd) != (B, N, d) or k.dtype != q.dtype or k.device != q.device:
        raise ValueError("key/value-side matrices must match the query side in B, N, d, dtype and device")
    if (Hkv == 0 and H != 0) or (Hkv > 0 and H % Hkv != 0):
        raise ValueError(f"the query heads ({H}) must be a multiple of the key/value heads ({Hkv})")
    _check_mats(*qside)
    _check_mats(*kside)
    return B, H, Hkv, N, d


def _check_rows(shape, *vs):
    for v in vs:
        if v.dtype != torch.float32 or tuple(v.shape) != tuple(shape[:3]) or not v.is_contiguous():
            raise ValueError("row vectors must be contiguous float32 [B, H, N]")


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream, like):
    """The stream to enqueue on: `stream`, or the current stream of the
    tensors' device.  The library launches on the current HIP device, which
    _call sets to the tensors' device, so the stream must belong to it too."""
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream(like.device).cuda_stream)
    if stream.device != like.device:
        raise ValueError(f"stream is on {stream.device} but the tensors are on {like.device}")
    return ctypes.c_void_p(stream.cuda_stream)


def _call(like, fn, *args):
    with torch.cuda.device(like.device):
        rc = fn(*args)
    if rc != BOB_OK:
        raise RuntimeError(status_string(rc))


def _column_workspace(query, code, B, H, Hkv, N, d, causal, columns, like, stream):
    """(workspace, bytes) for a *_ws call whose column blocks the library
    would split over workgroups (query: its bob_*_workspace_bytes), else
    (None, 0).  The fp32 partial sums go to a buffer from torch's allocator,
    kept from reuse until the kernels on `stream` are done."""
    with torch.cuda.device(like.device):
        nbytes = query(code, B, H, Hkv, N, d, causal, _opts(columns))
    if nbytes <= 0:
        return None, 0
    ws = torch.empty(nbytes, dtype=torch.uint8, device=like.device)
    if stream is not None:
        ws.record_stream(stream)
    return ws, nbytes


def _rows_empty(shape, like):
    return torch.empty(tuple(shape[:3]), dtype=torch.float32, device=like.device)


def attn_fwd_lse(Q, K, V, scale, causal=False, out=None, stream=None):
    """Forward attention (eq. 1): returns (O, L).  K, V may have fewer heads
    than Q (grouped-query attention, see include/flashbob.h)."""
    B, H, Hkv, N, d = _check_groups((Q,), (K, V))
    if out is None:
        out = (torch.empty_like(Q), _rows_empty(Q.shape, Q))
    O, L = out
    _check_mats(Q, O)
    _check_rows(Q.shape, L)
    lib = load_library()
    ptrs = (_p(Q), _p(K), _p(V), _p(O), _p(L), _stream(stream, Q))
    if Hkv == H:
        _call(Q, lib.attn_fwd_lse, _dtype_code(Q), B, H, N, d, float(scale), int(bool(causal)), *ptrs)
    else:
        _call(Q, lib.attn_fwd_lse_gqa, _dtype_code(Q), B, H, Hkv, N, d, float(scale), int(bool(causal)), *ptrs)
    return O, L


def attn_bwd(Q, K, V, O, dO, L, scale, causal=False, out=None, stream=None, columns=None):
    """First backward (eqs. 2-3): returns (dQ, dK, dV, D); dK, dV have K's shape.
    columns: ColumnOpts for the dK, dV kernel (None: automatic)."""
    B, H, Hkv, N, d = _check_groups((Q, O, dO), (K, V))
    _check_rows(Q.shape, L)
    if out is None:
        out = (torch.empty_like(Q), torch.empty_like(K), torch.empty_like(K), _rows_empty(Q.shape, Q))
    dQ, dK, dV, D = out
    _check_mats(Q, dQ)
    _check_mats(K, dK, dV)
    _check_rows(Q.shape, D)
    lib = load_library()
    code, c = _dtype_code(Q), int(bool(causal))
    ptrs = (_p(Q), _p(K), _p(V), _p(O), _p(dO), _p(L), _p(dQ), _p(dK), _p(dV), _p(D))
    st = _stream(stream, Q)
    ws, nbytes = _column_workspace(lib.bob_bwd_workspace_bytes, code, B, H, Hkv, N, d, c, columns, Q, stream)
    _call(Q, lib.attn_bwd_gqa_ws, code, B, H, Hkv, N, d, float(scale), c, *ptrs, _opts(columns),
          None if ws is None else _p(ws), nbytes, st)
    return dQ, dK, dV, D


def attn_bob_pass1_rows(Q, K, V, O, dO, gdQ, gdK, gdV, L, D, scale, causal=False, dQ=None, out=None,
                        stream=None):
    """BoB Pass 1 (row-major): returns (Qt, dOt, alpha, E).

    dQ (the first-backward output) is optional; when given, the kernel uses
    it in place of the R accumulator (see include/flashbob.h)."""
    B, H, Hkv, N, d = _check_groups((Q, O, dO, gdQ), (K, V, gdK, gdV))
    if dQ is not None:
        _check_mats(Q, dQ)
    _check_rows(Q.shape, L, D)
    if out is None:
        out = (torch.empty_like(Q), torch.empty_like(Q), _rows_empty(Q.shape, Q), _rows_empty(Q.shape, Q))
    Qt, dOt, alpha, E = out
    _check_mats(Q, Qt, dOt)
    _check_rows(Q.shape, alpha, E)
    lib = load_library()
    ptrs = (_p(Q), _p(K), _p(V), _p(O), _p(dO), _p(gdQ), _p(gdK), _p(gdV), _p(L), _p(D),
            None if dQ is None else _p(dQ), _p(Qt), _p(dOt), _p(alpha), _p(E), _stream(stream, Q))
    if Hkv == H:
        _call(Q, lib.attn_bob_pass1_rows, _dtype_code(Q), B, H, N, d, float(scale), int(bool(causal)), *ptrs)
    else:
        _call(Q, lib.attn_bob_pass1_rows_gqa, _dtype_code(Q), B, H, Hkv, N, d, float(scale), int(bool(causal)),
              *ptrs)
    return Qt, dOt, alpha, E


def attn_bob_pass2_cols(Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, scale, causal=False, out=None, stream=None,
                        columns=None):
    """BoB Pass 2 (column-major): returns (Kt, Vt), with K's shape.
    columns: ColumnOpts for its layout (None: automatic)."""
    B, H, Hkv, N, d = _check_groups((Q, dO, gdQ), (K, V, gdK, gdV))
    _check_rows(Q.shape, L, D, alpha, E)
    if out is None:
        out = (torch.empty_like(K), torch.empty_like(K))
    Kt, Vt = out
    _check_mats(K, Kt, Vt)
    lib = load_library()
    code, c = _dtype_code(Q), int(bool(causal))
    ptrs = (_p(Q), _p(K), _p(V), _p(dO), _p(gdQ), _p(gdK), _p(gdV), _p(L), _p(D), _p(alpha), _p(E),
            _p(Kt), _p(Vt))
    st = _stream(stream, Q)
    ws, nbytes = _column_workspace(lib.bob_pass2_workspace_bytes, code, B, H, Hkv, N, d, c, columns, Q, stream)
    _call(Q, lib.attn_bob_pass2_cols_gqa_ws, code, B, H, Hkv, N, d, float(scale), c, *ptrs, _opts(columns),
          None if ws is None else _p(ws), nbytes, st)
    return Kt, Vt


def attn_bob_pass2_cols_noalloc(Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, scale, causal=False, out=None,
                                stream=None, columns=None):
    """Pass 2 through attn_bob_pass2_cols_gqa_noalloc: a split layout keeps its
    partial sums in the library's static scratch buffer, so the call allocates
    no device memory (pass `out` to allocate nothing here either).  Calls that
    overlap on one device race on that buffer.  Returns (Kt, Vt)."""
    B, H, Hkv, N, d = _check_groups((Q, dO, gdQ), (K, V, gdK, gdV))
    _check_rows(Q.shape, L, D, alpha, E)
    if out is None:
        out = (torch.empty_like(K), torch.empty_like(K))
    Kt, Vt = out
    _check_mats(K, Kt, Vt)
    lib = load_library()
    ptrs = (_p(Q), _p(K), _p(V), _p(dO), _p(gdQ), _p(gdK), _p(gdV), _p(L), _p(D), _p(alpha), _p(E),
            _p(Kt), _p(Vt))
    _call(Q, lib.attn_bob_pass2_cols_gqa_noalloc, _dtype_code(Q), B, H, Hkv, N, d, float(scale),
          int(bool(causal)), *ptrs, _opts(columns), _stream(stream, Q))
    return Kt, Vt


def attn_bob3_alpha_rows(Q, K, gdQ, gdK, L, scale, causal=False, out=None, stream=None):
    """Three-pass control schedule, sweep 1: returns alpha."""
    B, H, N, d = _check_mats(Q, K, gdQ, gdK)
    _check_rows(Q.shape, L)
    alpha = _rows_empty(Q.shape, Q) if out is None else out
    _check_rows(Q.shape, alpha)
    lib = load_library()
    _call(Q, lib.attn_bob3_alpha_rows, _dtype_code(Q), B, H, N, d, float(scale), int(bool(causal)),
          _p(Q), _p(K), _p(gdQ), _p(gdK), _p(L), _p(alpha), _stream(stream, Q))
    return alpha


def attn_bob3_rows(Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, scale, causal=False, out=None, stream=None):
    """Three-pass control schedule, sweep 2: returns (Qt, dOt, E)."""
    B, H, N, d = _check_mats(Q, K, V, dO, gdQ, gdK, gdV)
    _check_rows(Q.shape, L, D, alpha)
    if out is None:
        out = (torch.empty_like(Q), torch.empty_like(Q), _rows_empty(Q.shape, Q))
    Qt, dOt, E = out
    _check_mats(Q, Qt, dOt)
    _check_rows(Q.shape, E)
    lib = load_library()
    _call(Q, lib.attn_bob3_rows, _dtype_code(Q), B, H, N, d, float(scale), int(bool(causal)),
          _p(Q), _p(K), _p(V), _p(dO), _p(gdQ), _p(gdK), _p(gdV), _p(L), _p(D), _p(alpha),
          _p(Qt), _p(dOt), _p(E), _stream(stream, Q))
    return Qt, dOt, E


def bob3(Q, K, V, dO, gdQ, gdK, gdV, scale, causal=False, stream=None, columns=None):
    """Whole path with the three-pass control schedule: forward, first
    backward, sweep 1 (alpha), sweep 2 (Qt, dOt, E), sweep 3 (Kt, Vt).
    Returns the same dict as bob()."""
    O, L = attn_fwd_lse(Q, K, V, scale, causal, stream=stream)
    dQ, dK, dV, D = attn_bwd(Q, K, V, O, dO, L, scale, causal, stream=stream, columns=columns)
    alpha = attn_bob3_alpha_rows(Q, K, gdQ, gdK, L, scale, causal, stream=stream)
    Qt, dOt, E = attn_bob3_rows(Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, scale, causal, stream=stream)
    Kt, Vt = attn_bob_pass2_cols(Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, scale, causal, stream=stream,
                                 columns=columns)
    return dict(Qt=Qt, Kt=Kt, Vt=Vt, dOt=dOt, alpha=alpha, E=E, O=O, L=L, D=D, dQ=dQ, dK=dK, dV=dV)


def bob(Q, K, V, dO, gdQ, gdK, gdV, scale, causal=False, use_dq=True, stream=None, columns=None):
    """Whole path: forward, first backward, Pass 1, Pass 2 on one stream.

    use_dq=True hands the first-backward dQ to Pass 1 (five-accumulator form);
    use_dq=False runs the six-accumulator form of Prop. 3.1.  columns: a
    ColumnOpts for both column kernels (None: automatic).

    Returns a dict with Qt, Kt, Vt, dOt, alpha, E and the producer state
    O, L, D, dQ, dK, dV.
    """
    O, L = attn_fwd_lse(Q, K, V, scale, causal, stream=stream)
    dQ, dK, dV, D = attn_bwd(Q, K, V, O, dO, L, scale, causal, stream=stream, columns=columns)
    Qt, dOt, alpha, E = attn_bob_pass1_rows(Q, K, V, O, dO, gdQ, gdK, gdV, L, D, scale, causal,
                                            dQ=dQ if use_dq else None, stream=stream)
    Kt, Vt = attn_bob_pass2_cols(Q, K, V, dO, gdQ, gdK, gdV, L, D, alpha, E, scale, causal, stream=stream,
                                 columns=columns)
    return dict(Qt=Qt, Kt=Kt, Vt=Vt, dOt=dOt, alpha=alpha, E=E, O=O, L=L, D=D, dQ=dQ, dK=dK, dV=dV)


from .autograd import attention  # noqa: E402  (differentiable wrapper; imports the entry points above)
