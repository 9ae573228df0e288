"""LoGra hot path on MI355X: thin Python binding of ``libpaper_logra.so``.

Each function has the name of the C entry point it calls (``include/logra.h``)
and only marshals arguments: torch device tensors become raw pointers, the
current torch stream becomes the HIP stream, and a non-OK status becomes a
``LograError``.  All computation happens in the HIP kernels.  The library must
have been built (``paper_2405_13954_amd.build.build()``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

__all__ = [
    "LograError", "lib", "F32", "BF16", "F64",
    "logra_version", "logra_last_error",
    "logra_project_ws_size", "logra_project_layer",
    "logra_project_layers_ws_size", "logra_project_layers",
    "logra_cov_accumulate", "logra_cov_accumulate_blocks", "logra_cov_accumulate_blocks_lower",
    "logra_cov_accumulate_f64",
    "logra_precondition_ws_size", "logra_precondition", "logra_precondition_blocks", "logra_precondition_f64",
    "logra_influence_ws_size", "logra_influence_scores",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpaper_logra.so")

F32, BF16, F64 = 0, 1, 2
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_HIP, ERR_NOT_PD, ERR_WORKSPACE, ERR_IO = 0, -1, -2, -3, -4, -5, -6
MAX_GROUP = 48
MAX_ACT_COV_GROUP = 32

EXPORTED = (
    "logra_last_error", "logra_version",
    "logra_project_ws_size", "logra_project_layer",
    "logra_project_layers_ws_size", "logra_project_layers", "logra_project_layers_noalloc",
    "logra_cov_accumulate", "logra_cov_accumulate_blocks", "logra_cov_accumulate_blocks_lower",
    "logra_cov_accumulate_f64",
    "logra_precondition_ws_size", "logra_precondition", "logra_precondition_blocks", "logra_precondition_f64",
    "logra_influence_ws_size", "logra_influence_scores", "logra_influence_scores_scaled",
    "logra_self_influence_ws_size", "logra_self_influence_blocks",
    "logra_act_cov_ws_size", "logra_act_cov_accumulate", "logra_act_cov_accumulate_group",
    "logra_pca_ws_size", "logra_pca_topk",
    "logra_influence_stream_ws_size", "logra_influence_stream", "logra_offload_rows",
    "logra_store_read_rows", "logra_store_write_rows", "logra_influence_stream_file_ws_size",
    "logra_influence_stream_file", "logra_offload_rows_file",
)


class LograError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"logra status {status}: {msg}")
        self.status = status


class LayerDesc(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("dy", ctypes.c_void_p), ("p_in", ctypes.c_void_p),
                ("p_out", ctypes.c_void_p), ("g_out", ctypes.c_void_p),
                ("n_in", ctypes.c_int), ("n_out", ctypes.c_int)]


class ActCovDesc(ctypes.Structure):
    """logra_act_cov_desc: one KFAC factor of a grouped SYRK launch."""
    _fields_ = [("a", ctypes.c_void_p), ("C", ctypes.c_void_p), ("n", ctypes.c_int)]


_lib = None


def lib():
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2405_13954_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz, f64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t, ctypes.c_double
        L.logra_last_error.restype = ctypes.c_char_p
        L.logra_version.restype = ctypes.c_char_p
        L.logra_project_ws_size.argtypes = [i32, i32, i32, i32, i32, i32]
        L.logra_project_ws_size.restype = sz
        L.logra_project_layer.argtypes = [vp, vp, i32, i32, i32, i32, i32, vp, vp, vp, i32, i32, vp, i32,
                                          i64, vp, sz, vp]
        L.logra_project_layers_ws_size.argtypes = [ctypes.POINTER(LayerDesc), i32, i32, i32, i32, i32]
        L.logra_project_layers_ws_size.restype = sz
        L.logra_project_layers.argtypes = [ctypes.POINTER(LayerDesc), i32, i32, i32, i32, vp, i32, i32,
                                           i32, i64, vp, sz, vp]
        L.logra_project_layers_noalloc.argtypes = [ctypes.POINTER(LayerDesc), i32, i32, i32, i32, vp, i32, i32,
                                                   i32, i64, vp]
        L.logra_cov_accumulate.argtypes = [vp, i32, i64, i32, i32, vp, vp]
        L.logra_cov_accumulate_blocks.argtypes = [vp, i32, i64, i32, i32, i32, vp, vp]
        L.logra_cov_accumulate_blocks_lower.argtypes = [vp, i32, i64, i32, i32, i32, vp, vp]
        L.logra_cov_accumulate_f64.argtypes = [vp, i32, i64, i32, i32, i32, vp, vp]
        L.logra_precondition_f64.argtypes = [vp, i32, i32, i64, f64, vp, i32, i64, i32, vp, i32, i64, vp, sz, vp]
        L.logra_precondition_ws_size.argtypes = [i32, i32, i32]
        L.logra_precondition_ws_size.restype = sz
        L.logra_precondition.argtypes = [vp, i32, i64, f64, vp, i32, i64, i32, vp, i32, i64, vp, sz, vp]
        L.logra_precondition_blocks.argtypes = [vp, i32, i32, i64, f64, vp, i32, i64, i32, vp, i32, i64,
                                                vp, sz, vp]
        L.logra_influence_ws_size.argtypes = [i32, i64, i32, i32]
        L.logra_influence_ws_size.restype = sz
        L.logra_influence_scores.argtypes = [vp, i32, i64, i32, vp, i32, i64, i64, i32, i64, vp, i64, i32,
                                             vp, vp, i32, vp, sz, vp]
        L.logra_influence_scores_scaled.argtypes = [vp, i32, i64, i32, vp, i32, i64, i64, i32, i64, vp, vp,
                                                    vp, i64, i32, vp, vp, i32, vp, sz, vp]
        L.logra_self_influence_ws_size.argtypes = [i32, i32]
        L.logra_self_influence_ws_size.restype = sz
        L.logra_self_influence_blocks.argtypes = [vp, i32, i32, i64, f64, vp, i32, i64, i64, vp, vp, vp, sz,
                                                  vp]
        L.logra_act_cov_ws_size.argtypes = [i32, i32]
        L.logra_act_cov_ws_size.restype = sz
        L.logra_act_cov_accumulate.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, sz, vp]
        L.logra_act_cov_accumulate_group.argtypes = [ctypes.POINTER(ActCovDesc), i32, i32, i32, i32, vp, vp, sz,
                                                     vp]
        L.logra_pca_ws_size.argtypes = [i32, i32]
        L.logra_pca_ws_size.restype = sz
        L.logra_pca_topk.argtypes = [vp, i32, i32, i32, vp, i32, i64, vp, vp, sz, vp]
        L.logra_influence_stream_ws_size.argtypes = [i32, i64, i32, i32, i32]
        L.logra_influence_stream_ws_size.restype = sz
        L.logra_influence_stream.argtypes = [vp, i32, i64, i32, vp, i32, i64, i64, i32, i64, i32, vp, vp, vp, sz,
                                             vp, vp]
        L.logra_offload_rows.argtypes = [vp, i64, vp, i64, i64, i64, vp, vp, vp]
        L.logra_store_read_rows.argtypes = [i32, i64, i64, i64, i64, vp, i64]
        L.logra_store_write_rows.argtypes = [i32, i64, i64, i64, i64, vp, i64]
        L.logra_influence_stream_file_ws_size.argtypes = [i32, i64, i32, i32, i32]
        L.logra_influence_stream_file_ws_size.restype = sz
        L.logra_influence_stream_file.argtypes = [vp, i32, i64, i32, i32, i64, i32, i64, i32, i64, i32, vp, vp, vp,
                                                  sz, vp, sz, vp, vp]
        L.logra_offload_rows_file.argtypes = [vp, i64, i64, i64, i32, i64, vp, sz, vp, vp, vp, vp]
        for name in ("logra_store_read_rows", "logra_store_write_rows", "logra_influence_stream_file",
                     "logra_offload_rows_file", "logra_offload_rows", "logra_influence_stream", "logra_pca_topk", "logra_act_cov_accumulate", "logra_act_cov_accumulate_group", "logra_project_layer", "logra_project_layers", "logra_project_layers_noalloc", "logra_cov_accumulate",
                     "logra_cov_accumulate_blocks", "logra_cov_accumulate_blocks_lower", "logra_precondition",
                     "logra_precondition_blocks",
                     "logra_cov_accumulate_f64", "logra_precondition_f64",
                     "logra_influence_scores", "logra_influence_scores_scaled", "logra_self_influence_blocks"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


# ------------------------------------------------------------------ helpers --
def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.float64:
        return F64
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16, float32 or float64)")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _event(done):
    """The hipEvent_t of a torch.cuda.Event (created by a first record if torch has not created it yet)."""
    if done is None:
        return None
    if not done.cuda_event:
        done.record()
    return ctypes.c_void_p(done.cuda_event)


def _check(rc: int):
    if rc != OK:
        raise LograError(rc, lib().logra_last_error().decode())


def _workspace(nbytes: int, device, ws=None):
    if nbytes == 0:
        return None, 0
    if ws is None:
        ws = _torch().empty(nbytes, dtype=_torch().uint8, device=device)
    return ws, ws.numel() * ws.element_size()


def _rows(t, width: int):
    """Row stride (elements) of a 2-D view whose rows are contiguous."""
    assert t.dim() == 2 and t.stride(1) == 1 and t.shape[1] >= width, "rows must be contiguous"
    return t.stride(0)


# --------------------------------------------------------------- entry points --
def logra_version() -> str:
    return lib().logra_version().decode()


def logra_last_error() -> str:
    return lib().logra_last_error().decode()


def logra_project_ws_size(B, T, n_in, n_out, k_in, k_out) -> int:
    return int(lib().logra_project_ws_size(B, T, n_in, n_out, k_in, k_out))


def logra_project_layers_ws_size(descs, n_layers, B, T, k_in, k_out) -> int:
    """descs: a ctypes array of LayerDesc (only n_in and n_out are read)."""
    return int(lib().logra_project_layers_ws_size(descs, n_layers, B, T, k_in, k_out))


def logra_project_layer(x, dy, p_in, p_out, g_out, mask=None, ws=None, stream=None):
    """G_b = sum_t m (P_out dy_bt)(P_in x_bt)^T into g_out rows (Sec. 3.1, Eq. (5)).

    x [B,T,n_in], dy [B,T,n_out], p_in [k_in,n_in], p_out [k_out,n_out] (same dtype),
    mask [B,T] uint8 or None, g_out [B, >=k_out*k_in] (a column slice of a store is fine).
    """
    B, T, n_in = x.shape
    n_out = dy.shape[2]
    k_in, k_out = p_in.shape[0], p_out.shape[0]
    g_ld = _rows(g_out, k_in * k_out) if B > 0 else k_in * k_out
    ws, wsb = _workspace(logra_project_ws_size(B, T, n_in, n_out, k_in, k_out), x.device, ws)
    _check(lib().logra_project_layer(_ptr(x), _ptr(dy), _dtype_code(x), B, T, n_in, n_out, _ptr(mask),
                                     _ptr(p_in), _ptr(p_out), k_in, k_out, _ptr(g_out), _dtype_code(g_out),
                                     g_ld, _ptr(ws), wsb, _stream(stream)))


def logra_project_layers(layers, mask=None, ws=None, stream=None):
    """Grouped projection of up to MAX_GROUP (48) layers of one batch.  layers: list of dicts with x, dy,
    p_in, p_out, g_out (shared B, T, k, dtypes and g_out row stride)."""
    n = len(layers)
    arr = (LayerDesc * n)()
    x0 = layers[0]["x"]
    B, T, _ = x0.shape
    k_in, k_out = layers[0]["p_in"].shape[0], layers[0]["p_out"].shape[0]
    g0 = layers[0]["g_out"]
    g_ld = _rows(g0, k_in * k_out) if B > 0 else k_in * k_out
    for i, L in enumerate(layers):
        arr[i] = LayerDesc(L["x"].data_ptr(), L["dy"].data_ptr(), L["p_in"].data_ptr(),
                           L["p_out"].data_ptr(), L["g_out"].data_ptr(), L["x"].shape[2], L["dy"].shape[2])
    ws, wsb = _workspace(logra_project_layers_ws_size(arr, n, B, T, k_in, k_out), x0.device, ws)
    _check(lib().logra_project_layers(arr, n, _dtype_code(x0), B, T, _ptr(mask), k_in, k_out,
                                      _dtype_code(g0), g_ld, _ptr(ws), wsb, _stream(stream)))


NOALLOC_WS_BYTES = 64 * 1024 * 1024


def logra_project_layers_noalloc(layers, mask=None, stream=None):
    """logra_project_layers with the library's static device workspace (no allocation;
    for callers that cannot allocate).  Same layer dicts as logra_project_layers."""
    n = len(layers)
    arr = (LayerDesc * n)()
    x0 = layers[0]["x"]
    B, T, _ = x0.shape
    k_in, k_out = layers[0]["p_in"].shape[0], layers[0]["p_out"].shape[0]
    g0 = layers[0]["g_out"]
    g_ld = _rows(g0, k_in * k_out) if B > 0 else k_in * k_out
    for i, L in enumerate(layers):
        arr[i] = LayerDesc(L["x"].data_ptr(), L["dy"].data_ptr(), L["p_in"].data_ptr(),
                           L["p_out"].data_ptr(), L["g_out"].data_ptr(), L["x"].shape[2], L["dy"].shape[2])
    _check(lib().logra_project_layers_noalloc(arr, n, _dtype_code(x0), B, T, _ptr(mask), k_in, k_out,
                                              _dtype_code(g0), g_ld, _stream(stream)))


def logra_cov_accumulate(g, S, stream=None):
    """S [D,D] fp32 += sum_b g_b g_b^T for g [B, D] (rows contiguous)."""
    B, D = g.shape
    ld = _rows(g, D) if B > 0 else D
    _check(lib().logra_cov_accumulate(_ptr(g), _dtype_code(g), ld, B, D, _ptr(S), _stream(stream)))


def logra_cov_accumulate_blocks(g, S, D: int, stream=None):
    """S [n_blocks, D, D] fp32; block l += G[:, l*D:(l+1)*D]^T G[:, l*D:(l+1)*D]."""
    B = g.shape[0]
    n_blocks = S.shape[0]
    ld = _rows(g, D * n_blocks) if B > 0 else D * n_blocks
    _check(lib().logra_cov_accumulate_blocks(_ptr(g), _dtype_code(g), ld, B, D, n_blocks, _ptr(S),
                                             _stream(stream)))


def logra_cov_accumulate_blocks_lower(g, S, D: int, stream=None):
    """S [n_blocks, D, D] fp32; the lower triangle (diagonal included) of block l
    += G[:, l*D:(l+1)*D]^T G[:, l*D:(l+1)*D]; entries above the diagonal untouched."""
    B = g.shape[0]
    n_blocks = S.shape[0]
    ld = _rows(g, D * n_blocks) if B > 0 else D * n_blocks
    _check(lib().logra_cov_accumulate_blocks_lower(_ptr(g), _dtype_code(g), ld, B, D, n_blocks, _ptr(S),
                                                   _stream(stream)))


def logra_cov_accumulate_f64(g, S, D: int = None, stream=None):
    """float64 statistic: S [D, D] or [n_blocks, D, D] fp64 += block-wise g^T g for g [B, n_blocks*D]
    (fp32 or fp64 rows)."""
    B = g.shape[0]
    n_blocks = 1 if S.dim() == 2 else S.shape[0]
    D = S.shape[-1] if D is None else D
    ld = _rows(g, D * n_blocks) if B > 0 else D * n_blocks
    _check(lib().logra_cov_accumulate_f64(_ptr(g), _dtype_code(g), ld, B, D, n_blocks, _ptr(S), _stream(stream)))


def logra_precondition_ws_size(D, n_blocks, Q) -> int:
    return int(lib().logra_precondition_ws_size(D, n_blocks, Q))


def logra_precondition(S, N: int, damp_ratio: float, g_test, g_out, ws=None, stream=None):
    """g_out[q] = (S/N + lambda I)^{-1} g_test[q], lambda = damp_ratio * tr(S/N)/D (synchronous)."""
    D = S.shape[0]
    Q = g_test.shape[0]
    ld_in = _rows(g_test, D) if Q > 0 else D
    ld_out = _rows(g_out, D) if Q > 0 else D
    ws, wsb = _workspace(logra_precondition_ws_size(D, 1, Q) if damp_ratio >= 0 else 0, S.device, ws)
    _check(lib().logra_precondition(_ptr(S), D, int(N), float(damp_ratio), _ptr(g_test), _dtype_code(g_test),
                                    ld_in, Q, _ptr(g_out), _dtype_code(g_out), ld_out, _ptr(ws), wsb,
                                    _stream(stream)))


def logra_precondition_blocks(S, N: int, damp_ratio: float, g_test, g_out, ws=None, stream=None):
    """Block-diagonal form: S [n_blocks, D, D]; g_test/g_out [Q, n_blocks*D]."""
    n_blocks, D, _ = S.shape
    Q = g_test.shape[0]
    ld_in = _rows(g_test, D * n_blocks) if Q > 0 else D * n_blocks
    ld_out = _rows(g_out, D * n_blocks) if Q > 0 else D * n_blocks
    ws, wsb = _workspace(logra_precondition_ws_size(D, n_blocks, Q) if damp_ratio >= 0 else 0, S.device, ws)
    _check(lib().logra_precondition_blocks(_ptr(S), D, n_blocks, int(N), float(damp_ratio), _ptr(g_test),
                                           _dtype_code(g_test), ld_in, Q, _ptr(g_out), _dtype_code(g_out),
                                           ld_out, _ptr(ws), wsb, _stream(stream)))


def logra_precondition_f64(S, N: int, damp_ratio: float, g_test, g_out, ws=None, stream=None):
    """logra_precondition_blocks with an fp64 S [D, D] or [n_blocks, D, D]; g_test / g_out may be
    fp32, bf16 or fp64 (synchronous)."""
    n_blocks = 1 if S.dim() == 2 else S.shape[0]
    D = S.shape[-1]
    Q = g_test.shape[0]
    ld_in = _rows(g_test, D * n_blocks) if Q > 0 else D * n_blocks
    ld_out = _rows(g_out, D * n_blocks) if Q > 0 else D * n_blocks
    ws, wsb = _workspace(logra_precondition_ws_size(D, n_blocks, Q) if damp_ratio >= 0 else 0, S.device, ws)
    _check(lib().logra_precondition_f64(_ptr(S), D, n_blocks, int(N), float(damp_ratio), _ptr(g_test),
                                        _dtype_code(g_test), ld_in, Q, _ptr(g_out), _dtype_code(g_out), ld_out,
                                        _ptr(ws), wsb, _stream(stream)))


def logra_influence_ws_size(Q, N_chunk, topk, scores_given) -> int:
    return int(lib().logra_influence_ws_size(Q, N_chunk, topk, int(bool(scores_given))))


def logra_influence_scores(g_test_pre, g_train, scores=None, topk: int = 0, topk_val=None,
                           topk_idx=None, train_base: int = 0, merge: bool = False, ws=None, stream=None,
                           row_scale=None, col_scale=None):
    """s = g_test_pre @ g_train^T (fp32) and/or the running per-query top-k.  With row_scale
    [Q] / col_scale [N] (fp32 device arrays), the scores and the top-k are those of
    s * row_scale[q] * col_scale[j] (logra_influence_scores_scaled)."""
    Q, D = g_test_pre.shape
    N = g_train.shape[0]
    ld_te = _rows(g_test_pre, D) if Q > 0 else D
    ld_tr = _rows(g_train, D) if N > 0 else D
    ld_s = _rows(scores, N) if scores is not None and Q > 0 else max(N, 1)
    ws, wsb = _workspace(logra_influence_ws_size(Q, N, topk, scores is not None), g_test_pre.device, ws)
    if row_scale is None and col_scale is None:
        _check(lib().logra_influence_scores(_ptr(g_test_pre), _dtype_code(g_test_pre), ld_te, Q, _ptr(g_train),
                                            _dtype_code(g_train), ld_tr, N, D, int(train_base), _ptr(scores),
                                            ld_s, int(topk), _ptr(topk_val), _ptr(topk_idx), int(bool(merge)),
                                            _ptr(ws), wsb, _stream(stream)))
    else:
        _check(lib().logra_influence_scores_scaled(_ptr(g_test_pre), _dtype_code(g_test_pre), ld_te, Q,
                                                   _ptr(g_train), _dtype_code(g_train), ld_tr, N, D,
                                                   int(train_base), _ptr(row_scale), _ptr(col_scale),
                                                   _ptr(scores), ld_s, int(topk), _ptr(topk_val),
                                                   _ptr(topk_idx), int(bool(merge)), _ptr(ws), wsb,
                                                   _stream(stream)))


def logra_self_influence_ws_size(D, n_blocks) -> int:
    return int(lib().logra_self_influence_ws_size(D, n_blocks))


def logra_self_influence_blocks(S, N: int, damp_ratio: float, g, self_out=None, rsqrt_out=None, ws=None,
                                stream=None):
    """self_j = sum_l g_jl^T (S_l/N + lambda_l I)^{-1} g_jl and/or 1/sqrt(self_j) for the rows of g
    [rows, n_blocks*D] (S [n_blocks, D, D] fp32)."""
    n_blocks, D, _ = S.shape
    rows = g.shape[0]
    ld = _rows(g, D * n_blocks) if rows > 0 else D * n_blocks
    ws, wsb = _workspace(logra_self_influence_ws_size(D, n_blocks), S.device, ws)
    _check(lib().logra_self_influence_blocks(_ptr(S), D, n_blocks, int(N), float(damp_ratio), _ptr(g),
                                             _dtype_code(g), ld, rows, _ptr(self_out), _ptr(rsqrt_out),
                                             _ptr(ws), wsb, _stream(stream)))


def logra_act_cov_ws_size(B, T) -> int:
    return int(lib().logra_act_cov_ws_size(B, T))


def logra_act_cov_accumulate(a, C, mask=None, ws=None, stream=None):
    """KFAC factor of one layer (Sec. 3.2): C [n, n] fp32 += sum over unmasked tokens of a_t a_t^T
    for a [B, T, n] (x for C_F, dy for C_B); mask [B, T] uint8 or None."""
    B, T, n = a.shape
    if B > 0 and T > 0:
        assert a.is_contiguous(), "a must be contiguous [B, T, n]"
    ws, wsb = _workspace(logra_act_cov_ws_size(B, T), C.device, ws)
    _check(lib().logra_act_cov_accumulate(_ptr(a), _dtype_code(a), B, T, n, _ptr(mask), _ptr(C), _ptr(ws), wsb,
                                          _stream(stream)))


def logra_act_cov_accumulate_group(factors, mask=None, ws=None, stream=None):
    """Several KFAC factors of one batch in one launch: factors is a list of
    (a [B, T, n_i], C [n_i, n_i] fp32) pairs sharing B, T, the dtype and the
    mask; each C += sum over unmasked tokens of a_t a_t^T, as
    logra_act_cov_accumulate would give it."""
    assert len(factors) > 0, "no factors"
    B, T, _ = factors[0][0].shape
    arr = (ActCovDesc * len(factors))()
    for i, (a, C) in enumerate(factors):
        assert a.shape[:2] == (B, T) and a.dtype == factors[0][0].dtype, "factors must share B, T and the dtype"
        if B > 0 and T > 0:
            assert a.is_contiguous(), "a must be contiguous [B, T, n]"
        arr[i] = ActCovDesc(_ptr(a), _ptr(C), a.shape[2])
    ws, wsb = _workspace(logra_act_cov_ws_size(B, T), factors[0][1].device, ws)
    _check(lib().logra_act_cov_accumulate_group(arr, len(factors), _dtype_code(factors[0][0]), B, T, _ptr(mask),
                                                _ptr(ws), wsb, _stream(stream)))


def logra_pca_ws_size(n, k) -> int:
    return int(lib().logra_pca_ws_size(n, k))


def logra_pca_topk(C, k: int, P, eigvals=None, iters: int = 30, ws=None, stream=None):
    """PCA initialisation (Sec. 3.2): rows of P [k, >= n] (fp32 or bf16) = the top-k eigenvectors
    of the symmetric fp32 C [n, n], by decreasing eigenvalue, sign rule as documented; eigvals
    [k] fp32 or None."""
    n = C.shape[0]
    ld_p = _rows(P, n)
    ws, wsb = _workspace(logra_pca_ws_size(n, k), C.device, ws)
    _check(lib().logra_pca_topk(_ptr(C), n, int(k), int(iters), _ptr(P), _dtype_code(P), ld_p, _ptr(eigvals),
                                _ptr(ws), wsb, _stream(stream)))


def logra_influence_stream_ws_size(Q, chunk_rows, D, tr_dtype, topk) -> int:
    return int(lib().logra_influence_stream_ws_size(Q, chunk_rows, D, tr_dtype, topk))


def logra_influence_stream(g_test_pre, g_train_host, topk: int, topk_val, topk_idx, chunk_rows: int, ws=None,
                           stream=None, copy_stream=None):
    """Running top-k of the scores of g_test_pre [Q, D] (device) against a store g_train_host
    [N, D] in pinned host memory (torch pin_memory=True), streamed in chunks of chunk_rows rows
    through two device staging buffers.  Synchronous."""
    Q, D = g_test_pre.shape
    N = g_train_host.shape[0]
    ld_te = _rows(g_test_pre, D) if Q > 0 else D
    ld_tr = _rows(g_train_host, D) if N > 0 else D
    code = _dtype_code(g_train_host)
    ws, wsb = _workspace(logra_influence_stream_ws_size(Q, chunk_rows, D, code, topk), g_test_pre.device, ws)
    cs = None if copy_stream is None else ctypes.c_void_p(copy_stream.cuda_stream)
    _check(lib().logra_influence_stream(_ptr(g_test_pre), _dtype_code(g_test_pre), ld_te, Q, _ptr(g_train_host),
                                        code, ld_tr, N, D, int(chunk_rows), int(topk), _ptr(topk_val),
                                        _ptr(topk_idx), _ptr(ws), wsb, _stream(stream), cs))


def logra_offload_rows(src, dst, stream=None, copy_stream=None, done=None):
    """Copy the rows of src [rows, w] (device) into dst [rows, w] (pinned host, torch pin_memory=True,
    same dtype) after the work enqueued on `stream`, on copy_stream (a torch.cuda.Stream) when given;
    done: an optional torch.cuda.Event recorded after the copy.  Asynchronous (App. E.2)."""
    rows = src.shape[0]
    if dst.shape[0] != rows or dst.shape[1] != src.shape[1] or dst.dtype != src.dtype:
        raise ValueError("src and dst must have the same rows, width and dtype")
    es = src.element_size()
    row_bytes = src.shape[1] * es
    ld_src = (_rows(src, src.shape[1]) if rows > 0 else src.shape[1]) * es
    ld_dst = (_rows(dst, dst.shape[1]) if rows > 0 else dst.shape[1]) * es
    cs = None if copy_stream is None else ctypes.c_void_p(copy_stream.cuda_stream)
    ev = _event(done)
    _check(lib().logra_offload_rows(_ptr(src), ld_src, _ptr(dst), ld_dst, rows, row_bytes, _stream(stream), cs, ev))


# ------------------------------------------------------------ store files --
def logra_store_write_rows(fd: int, file_offset: int, row0: int, rows):
    """Write the rows of a host numpy array (2-D, rows contiguous) as store rows row0.. of the file."""
    rows = np.ascontiguousarray(rows) if rows.strides[-1] != rows.itemsize else rows
    n = rows.shape[0]
    rb = rows.shape[1] * rows.itemsize
    _check(lib().logra_store_write_rows(int(fd), int(file_offset), int(row0), n, rb,
                                        rows.ctypes.data_as(ctypes.c_void_p) if n else None, rows.strides[0] if n else rb))


def logra_store_read_rows(fd: int, file_offset: int, row0: int, out):
    """Read store rows row0 .. row0 + len(out) - 1 of the file into the host numpy array out (2-D)."""
    n = out.shape[0]
    rb = out.shape[1] * out.itemsize
    _check(lib().logra_store_read_rows(int(fd), int(file_offset), int(row0), n, rb,
                                       out.ctypes.data_as(ctypes.c_void_p) if n else None, out.strides[0] if n else rb))


def logra_influence_stream_file_ws_size(Q, chunk_rows, D, tr_dtype, topk) -> int:
    return int(lib().logra_influence_stream_file_ws_size(Q, chunk_rows, D, tr_dtype, topk))


def logra_influence_stream_file(g_test_pre, fd: int, file_offset: int, N: int, D: int, tr_dtype: int, topk: int,
                                topk_val, topk_idx, chunk_rows: int, host_buf, ws=None, stream=None, copy_stream=None):
    """Running top-k of g_test_pre [Q, D] (device) against a store file of N rows of D elements of tr_dtype
    (F32, BF16 or F64 code), read by the library's reader thread into host_buf (a pinned uint8 tensor of at
    least 2 x round_up(chunk_rows x row bytes, 256) bytes).  Synchronous."""
    Q = g_test_pre.shape[0]
    ld_te = _rows(g_test_pre, D) if Q > 0 else D
    ws, wsb = _workspace(logra_influence_stream_file_ws_size(Q, chunk_rows, D, tr_dtype, topk), g_test_pre.device, ws)
    cs = None if copy_stream is None else ctypes.c_void_p(copy_stream.cuda_stream)
    _check(lib().logra_influence_stream_file(_ptr(g_test_pre), _dtype_code(g_test_pre), ld_te, Q, int(fd),
                                             int(file_offset), int(tr_dtype), int(N), int(D), int(chunk_rows),
                                             int(topk), _ptr(topk_val), _ptr(topk_idx), _ptr(host_buf),
                                             host_buf.numel() * host_buf.element_size(), _ptr(ws), wsb,
                                             _stream(stream), cs))


def logra_offload_rows_file(src, fd: int, file_offset: int, host_buf, io_status=None, stream=None, copy_stream=None,
                            done=None):
    """Write-behind of the device rows src [rows, w] to the store file at file_offset through the pinned
    host_buf (uint8 tensor); io_status: a ctypes.c_int set to 1, then 0 or ERR_IO once written."""
    rows = src.shape[0]
    es = src.element_size()
    row_bytes = src.shape[1] * es
    ld_src = (_rows(src, src.shape[1]) if rows > 0 else src.shape[1]) * es
    cs = None if copy_stream is None else ctypes.c_void_p(copy_stream.cuda_stream)
    ev = _event(done)
    st = None if io_status is None else ctypes.byref(io_status)
    _check(lib().logra_offload_rows_file(_ptr(src), ld_src, rows, row_bytes, int(fd), int(file_offset), _ptr(host_buf),
                                         host_buf.numel() * host_buf.element_size(), st, _stream(stream), cs, ev))
