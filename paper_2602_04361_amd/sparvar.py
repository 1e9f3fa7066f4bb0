"""ctypes binding of libsparvar.so (argument marshalling only).

Every function here has the name of the C entry point it calls and forwards
torch tensors as raw device pointers, plane strides and the current HIP stream.
No computation happens in Python. If the shared library is missing the first
call raises: there is no fallback path.
"""
from __future__ import annotations

import contextlib
import ctypes
import math
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# SPARVAR_LIBRARY selects another build of the same library (e.g. the
# host-sanitized one of build_host_sanitized.py); the default is the in-tree build.
LIB_PATH = os.environ.get("SPARVAR_LIBRARY") or os.path.join(_HERE, "libsparvar.so")

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_CAPACITY, ERR_HIP = 0, -1, -2, -3, -4
BF16, F32 = 0, 1
MAX_SCALES = 32
NOALLOC_MAX_ROWS = 1 << 20  # SPARVAR_NOALLOC_MAX_ROWS

EXPORTS = [
    "sparvar_scale_info",
    "sparvar_dense_attn_fwd",
    "sparvar_select_blocks",
    "sparvar_decision_step",
    "sparvar_cs4a_column_sums",
    "sparvar_cs4a_select_tokens",
    "sparvar_cs4a_row_stride",
    "sparvar_cs4a_map_tokens",
    "sparvar_cs4a_attn_fwd",
    "sparvar_map_index_steps",
    "sparvar_map_index_steps_noalloc",
    "sparvar_kv_compact",
    "sparvar_csla_row_stride",
    "sparvar_csla_block_rows",
    "sparvar_csla_attn_fwd",
    "sparvar_local_blocks_capacity",
    "sparvar_local_blocks",
    "sparvar_map_index_capacity",
    "sparvar_map_index",
    "sparvar_block_sparse_attn_fwd",
    "sparvar_status_string",
    "sparvar_last_error",
    "sparvar_set_launch_option",
    "sparvar_get_launch_option",
]

# sparvar_launch_option_t, in enum order
LAUNCH_OPTIONS = ["SWIZZLE", "DENSE_WAVES", "DENSE_CHUNK", "DENSE_STAGES", "SPARSE_WAVES", "SPARSE_CHUNK",
                  "SPARSE_STAGES", "SPARSE_GROUP_WAVES", "SPARSE_GROUP_CHUNK", "SPARSE_GROUP_STAGES", "CSLA_CHUNK",
                  "CSLA_STAGES", "CS4A_CHUNK", "DECISION_FUSED"]
OPT_DEFAULT = -(1 << 31)
# sparvar_projection_t
PROJECT_POINT, PROJECT_COVER = 0, 1
PROJECTIONS = {"point": PROJECT_POINT, "cover": PROJECT_COVER, PROJECT_POINT: PROJECT_POINT,
               PROJECT_COVER: PROJECT_COVER}


class SparvarError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{message} (status {status})")
        self.status = status


class _CGeometry(ctypes.Structure):
    _fields_ = [
        ("num_scales", ctypes.c_int32),
        ("h", ctypes.POINTER(ctypes.c_int32)),
        ("w", ctypes.POINTER(ctypes.c_int32)),
        ("block_edge", ctypes.c_int32),
        ("num_sink_scales", ctypes.c_int32),
    ]


class _CScaleInfo(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "h", "w", "n_tokens", "token_offset", "n_tokens_le", "tile_h", "tile_w",
        "tiles_h", "tiles_w", "block_offset", "n_blocks_le")]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libsparvar.so once and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2602_04361_amd.build`")
    lib = ctypes.CDLL(path)
    i32, i64, f32, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
    G = ctypes.POINTER(_CGeometry)
    sig = {
        "sparvar_scale_info": (ctypes.c_int, [G, i32, ctypes.POINTER(_CScaleInfo)]),
        "sparvar_dense_attn_fwd": (ctypes.c_int, [i32, i32, i32, i32, i32, ctypes.c_int, vp, i64, vp, vp, i64, vp,
                                                  vp, f32, vp]),
        "sparvar_select_blocks": (ctypes.c_int, [G, i32, i32, i32, i32, ctypes.c_int, vp, i64, vp, i64, vp, f32, vp,
                                                 vp, i32, vp, vp]),
        "sparvar_decision_step": (ctypes.c_int, [G, i32, i32, i32, i32, ctypes.c_int, vp, i64, vp, vp, i64, vp, vp,
                                                 f32, vp, i32, vp, vp]),
        "sparvar_cs4a_column_sums": (ctypes.c_int, [G, i32, i32, i32, i32, i32, ctypes.c_int, vp, i64, vp, i64, vp,
                                                    f32, vp, vp]),
        "sparvar_cs4a_select_tokens": (ctypes.c_int, [vp, i32, i32, i32, vp, vp]),
        "sparvar_cs4a_row_stride": (i32, [G, i32]),
        "sparvar_map_index_steps": (ctypes.c_int, [G, i32, i32, vp, i32, i32, i32, vp, i32, i32, i32, vp, vp, vp,
                                                   vp, vp]),
        "sparvar_map_index_steps_noalloc": (ctypes.c_int, [G, i32, i32, vp, i32, i32, i32, vp, i32, i32, i32, vp, vp,
                                                           vp, vp, vp]),
        "sparvar_kv_compact": (ctypes.c_int, [G, i32, vp, i32, i32, i32, ctypes.c_int, vp, vp, i64, vp, vp, i64, vp]),
        "sparvar_csla_row_stride": (i32, [G, i32, i32]),
        "sparvar_csla_block_rows": (ctypes.c_int, [G, i32, vp, i32, vp, i32, vp]),
        "sparvar_csla_attn_fwd": (ctypes.c_int, [G, i32, i32, i32, i32, i32, ctypes.c_int, vp, i64, vp, vp, i64, vp,
                                                 vp, ctypes.c_float, vp, i32, vp]),
        "sparvar_cs4a_map_tokens": (ctypes.c_int, [G, i32, i32, i32, i32, i32, i32, vp, vp, i32, vp]),
        "sparvar_cs4a_attn_fwd": (ctypes.c_int, [G, i32, i32, i32, i32, i32, ctypes.c_int, vp, i64, vp, vp, i64, vp,
                                                 vp, f32, vp, i32, i32, vp, i32, vp]),
        "sparvar_local_blocks_capacity": (i64, [G, i32, i32, i32]),
        "sparvar_local_blocks": (ctypes.c_int, [G, i32, i32, i32, vp, vp, i64, vp]),
        "sparvar_map_index_capacity": (i64, [G, i32, i32, i32, i32, i32, i32, i32, i32]),
        "sparvar_map_index": (ctypes.c_int, [G, i32, i32, i32, i32, i32, vp, vp, vp, i32, i32, i32, vp, vp, i64, vp,
                                             vp, vp]),
        "sparvar_block_sparse_attn_fwd": (ctypes.c_int, [G, i32, i32, i32, i32, ctypes.c_int, vp, i64, vp, vp, i64,
                                                         vp, vp, f32, vp, vp, vp, vp]),
        "sparvar_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "sparvar_last_error": (ctypes.c_char_p, []),
        "sparvar_set_launch_option": (ctypes.c_int, [i32, i32]),
        "sparvar_get_launch_option": (ctypes.c_int, [i32, ctypes.POINTER(ctypes.c_int32)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status):
    if status != OK:
        lib = load_library()
        raise SparvarError(status, lib.sparvar_last_error().decode() or lib.sparvar_status_string(status).decode())


class Geometry:
    """Host-side sparvar_geometry_t: scale sizes, block edge, sink scales."""

    def __init__(self, h, w, block_edge, num_sink_scales):
        self.h = [int(x) for x in h]
        self.w = [int(x) for x in w]
        self.block_edge = int(block_edge)
        self.num_sink_scales = int(num_sink_scales)
        n = len(self.h)
        self._h = (ctypes.c_int32 * n)(*self.h)
        self._w = (ctypes.c_int32 * n)(*self.w)
        self.c = _CGeometry(n, self._h, self._w, self.block_edge, self.num_sink_scales)

    @property
    def ref(self):
        return ctypes.byref(self.c)

    def scale_info(self, l):
        info = _CScaleInfo()
        _check(load_library().sparvar_scale_info(self.ref, int(l), ctypes.byref(info)))
        return {n: getattr(info, n) for n, _ in _CScaleInfo._fields_}


def sparvar_set_launch_option(name, value=None):
    """Set launch option `name` (a LAUNCH_OPTIONS entry) process-wide; None restores its default."""
    _check(load_library().sparvar_set_launch_option(LAUNCH_OPTIONS.index(name),
                                                    OPT_DEFAULT if value is None else int(value)))


def sparvar_get_launch_option(name):
    v = ctypes.c_int32()
    _check(load_library().sparvar_get_launch_option(LAUNCH_OPTIONS.index(name), ctypes.byref(v)))
    return v.value


@contextlib.contextmanager
def launch_options(**opts):
    """Set launch options for the body of a with-statement, then restore the previous values."""
    before = {n: sparvar_get_launch_option(n) for n in opts}
    try:
        for n, v in opts.items():
            sparvar_set_launch_option(n, v)
        yield
    finally:
        for n, v in before.items():
            sparvar_set_launch_option(n, v)


# ---------------------------------------------------------------- tensor helpers
def _torch():
    import torch  # imported lazily so that the geometry helpers work without torch

    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise SparvarError(ERR_UNSUPPORTED, f"dtype {t.dtype} not supported")


def _plane_stride(t, name):
    """[B,H,rows,d] tensor with d and rows contiguous and evenly spaced planes."""
    if t.dim() != 4:
        raise SparvarError(ERR_INVALID, f"{name} must be [B,H,rows,d]")
    B, H, _, d = t.shape
    if t.stride(3) != 1 or t.stride(2) != d:
        raise SparvarError(ERR_INVALID, f"{name} rows must be contiguous")
    if B > 1 and t.stride(0) != H * t.stride(1):
        raise SparvarError(ERR_INVALID, f"{name} planes must be evenly spaced")
    return t.stride(1)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = _torch().cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _scale(softmax_scale, d):
    return float(1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale)


# ---------------------------------------------------------------- entry points
def sparvar_dense_attn_fwd(q, k, v, o, lse=None, softmax_scale=None, stream=None):
    """O = softmax(scale Q K^T) V over all keys; see sparvar.h."""
    lib = load_library()
    B, H, n_q, d = q.shape
    n_kv = k.shape[2]
    if _plane_stride(v, "v") != _plane_stride(k, "k"):
        raise SparvarError(ERR_INVALID, "k and v must share one plane stride")
    _check(lib.sparvar_dense_attn_fwd(B, H, n_q, n_kv, d, _dtype_code(q), _ptr(q), _plane_stride(q, "q"),
                                      _ptr(k), _ptr(v), _plane_stride(k, "k"), _ptr(o), _ptr(lse),
                                      _scale(softmax_scale, d), _stream(stream)))
    return o, lse


def sparvar_select_blocks(geom, S, q_S, k_leS, lse_S, topk, topk_idx, scores_out=None, scores_in=None,
                          softmax_scale=None, B=None, H=None, d=None, stream=None):
    """Decision-scale pooled scores and per-query-tile top-k; see sparvar.h."""
    lib = load_library()
    if scores_in is None:
        B, H, _, d = q_S.shape
        dt = _dtype_code(q_S)
        qs, ks = _plane_stride(q_S, "q_S"), _plane_stride(k_leS, "k_leS")
    else:
        B, H = scores_in.shape[0], scores_in.shape[1]
        d = 128 if d is None else d
        dt, qs, ks = BF16, 0, 0
    _check(lib.sparvar_select_blocks(geom.ref, S, B, H, d, dt, _ptr(q_S), qs, _ptr(k_leS), ks, _ptr(lse_S),
                                     _scale(softmax_scale, d), _ptr(scores_in), _ptr(scores_out), topk,
                                     _ptr(topk_idx), _stream(stream)))
    return topk_idx


def sparvar_decision_step(geom, S, q_S, k_leS, v_leS, o_S, lse_S, scores_out, topk, topk_idx, softmax_scale=None,
                          stream=None):
    """Dense attention + LSE, pooled scores and top-k at the decision scale; see sparvar.h."""
    lib = load_library()
    B, H, _, d = q_S.shape
    if _plane_stride(v_leS, "v_leS") != _plane_stride(k_leS, "k_leS"):
        raise SparvarError(ERR_INVALID, "k_leS and v_leS must share one plane stride")
    _check(lib.sparvar_decision_step(geom.ref, S, B, H, d, _dtype_code(q_S), _ptr(q_S), _plane_stride(q_S, "q_S"),
                                     _ptr(k_leS), _ptr(v_leS), _plane_stride(k_leS, "k_leS"), _ptr(o_S), _ptr(lse_S),
                                     _scale(softmax_scale, d), _ptr(scores_out), topk, _ptr(topk_idx),
                                     _stream(stream)))
    return topk_idx


def sparvar_cs4a_column_sums(geom, S, C, q_S, k_leS, lse_S, colsum, softmax_scale=None, stream=None):
    """Token column sums over 1-D query blocks of C queries at S; see sparvar.h."""
    lib = load_library()
    B, H, _, d = q_S.shape
    _check(lib.sparvar_cs4a_column_sums(geom.ref, S, C, B, H, d, _dtype_code(q_S), _ptr(q_S), _plane_stride(q_S, "q_S"),
                                        _ptr(k_leS), _plane_stride(k_leS, "k_leS"), _ptr(lse_S),
                                        _scale(softmax_scale, d), _ptr(colsum), _stream(stream)))
    return colsum


def sparvar_cs4a_select_tokens(values, K, inds, stream=None):
    """Top-K per row of values [..., n] into inds [..., K]; see sparvar.h."""
    n = values.shape[-1]
    rows = values.numel() // n
    if not values.is_contiguous() or not inds.is_contiguous() or inds.numel() != rows * K:
        raise SparvarError(ERR_INVALID, "values and inds must be contiguous [rows, n] and [rows, K]")
    _check(load_library().sparvar_cs4a_select_tokens(_ptr(values), rows, n, K, _ptr(inds), _stream(stream)))
    return inds


def sparvar_cs4a_row_stride(geom, K):
    m = load_library().sparvar_cs4a_row_stride(geom.ref, K)
    if m < 0:
        _check(int(m))
    return int(m)


def sparvar_cs4a_map_tokens(geom, S, k, C, B, H, K, inds_S, tokens, M, stream=None):
    """Sink tokens + mapped top-K tokens for every query block of scale k; see sparvar.h."""
    _check(load_library().sparvar_cs4a_map_tokens(geom.ref, S, k, C, B, H, K, _ptr(inds_S), _ptr(tokens), M,
                                                  _stream(stream)))
    return tokens


def sparvar_cs4a_attn_fwd(geom, k, C, q_k, k_lek, v_lek, o, tokens, M, lse=None, mode=0, base=None, base_scale=0,
                          softmax_scale=None, stream=None):
    """Gather attention over token rows (mode 0), O_cache (1) or O_cache upsampled + sparse update (2)."""
    lib = load_library()
    B, H, _, d = q_k.shape
    if _plane_stride(v_lek, "v_lek") != _plane_stride(k_lek, "k_lek"):
        raise SparvarError(ERR_INVALID, "k_lek and v_lek must share one plane stride")
    _check(lib.sparvar_cs4a_attn_fwd(geom.ref, k, C, B, H, d, _dtype_code(q_k), _ptr(q_k), _plane_stride(q_k, "q_k"),
                                     _ptr(k_lek), _ptr(v_lek), _plane_stride(k_lek, "k_lek"), _ptr(o), _ptr(lse),
                                     _scale(softmax_scale, d), _ptr(tokens), M, mode, _ptr(base), base_scale,
                                     _stream(stream)))
    return o


def sparvar_kv_compact(geom, keep, k_src, v_src, k_dst, v_dst, stream=None):
    """Copy the K/V tokens of the kept scales (1-based, ascending) into a compact cache; see sparvar.h."""
    B, H, _, d = k_src.shape
    if _plane_stride(v_src, "v_src") != _plane_stride(k_src, "k_src") or \
            _plane_stride(v_dst, "v_dst") != _plane_stride(k_dst, "k_dst"):
        raise SparvarError(ERR_INVALID, "K and V must share plane strides")
    arr = (ctypes.c_int32 * max(len(keep), 1))(*[int(l) for l in keep])
    _check(load_library().sparvar_kv_compact(geom.ref, len(keep), ctypes.cast(arr, ctypes.c_void_p), B, H, d,
                                             _dtype_code(k_src), _ptr(k_src), _ptr(v_src),
                                             _plane_stride(k_src, "k_src"), _ptr(k_dst), _ptr(v_dst),
                                             _plane_stride(k_dst, "k_dst"), _stream(stream)))
    return k_dst, v_dst


def compact_geometry(geom, keep, num_sink_scales=None):
    """Geometry of the compact cache that keeps scales `keep` (its scales are the kept ones, in order)."""
    keep = [int(l) for l in keep]
    ns = geom.num_sink_scales if num_sink_scales is None else num_sink_scales
    return Geometry([geom.h[l - 1] for l in keep], [geom.w[l - 1] for l in keep], geom.block_edge, ns)


def sparvar_csla_row_stride(geom, k, block):
    m = load_library().sparvar_csla_row_stride(geom.ref, k, block)
    if m < 0:
        _check(int(m))
    return int(m)


def sparvar_csla_block_rows(geom, k, windows, block, rows, stream=None):
    """CSLA key-block rows of every 1-D query block of scale k (windows: one size per scale 1..k); see sparvar.h."""
    win = (ctypes.c_int32 * max(len(windows), 1))(*[int(w) for w in windows])
    if len(windows) != k:
        raise SparvarError(ERR_INVALID, "one window size per scale 1..k is required")
    _check(load_library().sparvar_csla_block_rows(geom.ref, k, ctypes.cast(win, ctypes.c_void_p), block, _ptr(rows),
                                                  rows.shape[-1], _stream(stream)))
    return rows


def sparvar_csla_attn_fwd(geom, k, block, q_k, k_lek, v_lek, o, rows, lse=None, softmax_scale=None, stream=None):
    """Block-sparse attention of scale k over CSLA block rows (shared by every head)."""
    lib = load_library()
    B, H, _, d = q_k.shape
    if _plane_stride(v_lek, "v_lek") != _plane_stride(k_lek, "k_lek"):
        raise SparvarError(ERR_INVALID, "k_lek and v_lek must share one plane stride")
    _check(lib.sparvar_csla_attn_fwd(geom.ref, k, block, B, H, d, _dtype_code(q_k), _ptr(q_k),
                                     _plane_stride(q_k, "q_k"), _ptr(k_lek), _ptr(v_lek), _plane_stride(k_lek, "k_lek"),
                                     _ptr(o), _ptr(lse), _scale(softmax_scale, d), _ptr(rows), rows.shape[-1],
                                     _stream(stream)))
    return o


def sparvar_local_blocks_capacity(geom, k, radius, prev_dilation=0):
    n = load_library().sparvar_local_blocks_capacity(geom.ref, k, radius, prev_dilation)
    if n < 0:
        _check(int(n))
    return int(n)


def sparvar_local_blocks(geom, k, radius, row_ptr, col_idx, prev_dilation=0, stream=None):
    _check(load_library().sparvar_local_blocks(geom.ref, k, radius, prev_dilation, _ptr(row_ptr), _ptr(col_idx),
                                               col_idx.numel(), _stream(stream)))
    return row_ptr, col_idx


def sparvar_map_index_capacity(geom, S, k, B, H, topk, radius, prev_dilation=0, projection=PROJECT_POINT):
    n = load_library().sparvar_map_index_capacity(geom.ref, S, k, B, H, topk, radius, prev_dilation,
                                                  PROJECTIONS[projection])
    if n < 0:
        _check(int(n))
    return int(n)


def sparvar_map_index(geom, S, k, B, H, topk, topk_idx, local_row_ptr, local_col_idx, radius, row_ptr, col_idx,
                      schedule=None, prev_dilation=0, status=None, projection=PROJECT_POINT, stream=None):
    """Mapped + local blocks -> CSR; local_row_ptr/local_col_idx may both be None. status (optional one-element
    int32 device tensor, cleared by the caller) receives ERR_CAPACITY if a supplied local row was cut."""
    _check(load_library().sparvar_map_index(geom.ref, S, k, B, H, topk, _ptr(topk_idx), _ptr(local_row_ptr),
                                            _ptr(local_col_idx), radius, prev_dilation, PROJECTIONS[projection],
                                            _ptr(row_ptr),
                                            _ptr(col_idx), col_idx.numel(), _ptr(schedule), _ptr(status),
                                            _stream(stream)))
    return row_ptr, col_idx, schedule


def sparvar_map_index_steps(geom, S, ks, B, H, topk, topk_idx, radius, row_ptrs, col_idxs, prev_dilation=0,
                            orders=None, projection=PROJECT_POINT, stream=None, noalloc=False):
    """The rows of several target scales in one launch (local rows generated); with orders (one int32 tensor of
    B*H*G_k entries, or None, per step) also the attention launch order of each step. noalloc=True calls
    sparvar_map_index_steps_noalloc (row lengths in the library's fixed scratch; col_idxs need only the row
    slots)."""
    n = len(ks)
    if not (len(row_ptrs) == len(col_idxs) == n):
        raise SparvarError(ERR_INVALID, "one row_ptr and col_idx per step is required")
    k_arr = (ctypes.c_int32 * max(n, 1))(*[int(k) for k in ks])
    rp_arr = (ctypes.c_void_p * max(n, 1))(*[t.data_ptr() for t in row_ptrs])
    ci_arr = (ctypes.c_void_p * max(n, 1))(*[t.data_ptr() for t in col_idxs])
    cap_arr = (ctypes.c_int64 * max(n, 1))(*[t.numel() for t in col_idxs])
    vp = ctypes.c_void_p
    ord_arr = None
    if orders is not None:
        if len(orders) != n:
            raise SparvarError(ERR_INVALID, "one order (or None) per step is required")
        ord_arr = (ctypes.c_void_p * max(n, 1))(*[(t.data_ptr() if t is not None else None) for t in orders])
    lib = load_library()
    fn = lib.sparvar_map_index_steps_noalloc if noalloc else lib.sparvar_map_index_steps
    _check(fn(geom.ref, S, n, ctypes.cast(k_arr, vp), B, H, topk, _ptr(topk_idx), radius, prev_dilation,
              PROJECTIONS[projection], ctypes.cast(rp_arr, vp), ctypes.cast(ci_arr, vp), ctypes.cast(cap_arr, vp),
              ctypes.cast(ord_arr, vp) if ord_arr is not None else None, _stream(stream)))


def sparvar_block_sparse_attn_fwd(geom, k, q_k, k_lek, v_lek, o, row_ptr, col_idx, lse=None, schedule=None,
                                  softmax_scale=None, stream=None):
    """Block-sparse attention of scale-k queries over the kept blocks; see sparvar.h."""
    lib = load_library()
    B, H, _, d = q_k.shape
    if _plane_stride(v_lek, "v_lek") != _plane_stride(k_lek, "k_lek"):
        raise SparvarError(ERR_INVALID, "k_lek and v_lek must share one plane stride")
    _check(lib.sparvar_block_sparse_attn_fwd(geom.ref, k, B, H, d, _dtype_code(q_k), _ptr(q_k),
                                             _plane_stride(q_k, "q_k"), _ptr(k_lek), _ptr(v_lek),
                                             _plane_stride(k_lek, "k_lek"), _ptr(o), _ptr(lse),
                                             _scale(softmax_scale, d), _ptr(row_ptr), _ptr(col_idx),
                                             _ptr(schedule), _stream(stream)))
    return o, lse
