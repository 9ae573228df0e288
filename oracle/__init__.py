"""LoGra float64 CPU oracle -- test infrastructure, not part of the product.

Thin numpy wrappers over ``logra_oracle.c``: a plain, slow float64
implementation of what the LoGra hot path computes (arXiv 2405.13954,
Sec. 2 Eq. (2)-(3), Sec. 3.1 Eq. (4)-(5), Sec. 3.2 (the KFAC-eigenvector
initialisation of the projections), Sec. 4.2 (l-RelatIF), App. C and App. D).
The PCA step takes numpy's float64 eigh as its eigendecomposition.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import this
package; the product path never does, and this package imports nothing from
it.

Array conventions: numpy arrays on the host; bf16 data is carried as uint16
bit patterns, fp32 as float32, fp64 as float64.  Outputs are float64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "logra_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liblogra_oracle.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_NOT_PD = -4

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (C99, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-std=c99", "-O2", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
               _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        # LOGRA_ORACLE_LIB points the tests at a deliberately broken build of
        # this file (the mutation test); normally unset.
        path = os.environ.get("LOGRA_ORACLE_LIB")
        if not path:
            path = _LIB_PATH
            if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
                build(force=True)
        L = ctypes.CDLL(path)
        vp, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
        proj = [vp, vp, i32, i32, i32, i32, i32, vp, vp, vp, i32, i32, vp]
        L.oracle_project_factored.argtypes = proj
        L.oracle_project_dense.argtypes = proj
        L.oracle_project_factored_layers.argtypes = [i32, vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, i32, i32, vp]
        L.oracle_cov_accumulate.argtypes = [vp, i32, i64, i32, i32, vp]
        L.oracle_precondition.argtypes = [vp, i32, i64, f64, vp, i32, i64, i32, vp, i64, vp]
        L.oracle_scores.argtypes = [vp, i32, i64, i32, vp, i32, i64, i64, i32, vp, i64]
        L.oracle_topk.argtypes = [vp, i64, i32, i64, i64, i32, vp, vp]
        L.oracle_self_influence.argtypes = [vp, i32, i64, f64, vp, i32, i64, i32, vp]
        L.oracle_normalise_scores.argtypes = [vp, i64, i32, i64, vp, vp]
        L.oracle_act_cov.argtypes = [vp, i32, i32, i32, i32, vp, vp]
        L.oracle_num_threads.argtypes = []
        for name in ("oracle_project_factored", "oracle_project_factored_layers", "oracle_project_dense",
                     "oracle_cov_accumulate",
                     "oracle_precondition", "oracle_scores", "oracle_topk", "oracle_self_influence",
                     "oracle_normalise_scores", "oracle_act_cov", "oracle_num_threads"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return 0
    if a.dtype == np.uint16:
        return 1
    if a.dtype == np.float64:
        return 2
    raise TypeError(f"oracle: unsupported dtype {a.dtype}")


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a):
    return None if a is None else np.ascontiguousarray(a)


def _check(rc: int, what: str):
    if rc == ERR_NOT_PD:
        raise np.linalg.LinAlgError(f"{what}: matrix is not positive definite")
    if rc != OK:
        raise ValueError(f"{what}: status {rc}")


def _project(fn, x, dy, p_in, p_out, mask=None):
    x, dy, p_in, p_out, mask = map(_c, (x, dy, p_in, p_out, mask))
    B, T, n_in = x.shape
    n_out = dy.shape[2]
    k_in, k_out = p_in.shape[0], p_out.shape[0]
    code = _code(x)
    assert _code(dy) == code and _code(p_in) == code and _code(p_out) == code
    assert dy.shape[:2] == (B, T) and p_in.shape[1] == n_in and p_out.shape[1] == n_out
    if mask is not None:
        mask = mask.astype(np.uint8, copy=False)
        assert mask.shape == (B, T)
    g = np.zeros((B, k_out * k_in), dtype=np.float64)
    rc = fn(_ptr(x), _ptr(dy), code, B, T, n_in, n_out, _ptr(mask), _ptr(p_in), _ptr(p_out),
            k_in, k_out, _ptr(g))
    _check(rc, fn.__name__)
    return g


def project_factored(x, dy, p_in, p_out, mask=None) -> np.ndarray:
    """Eq. (5) right side: G_b = sum_t (P_out dy_t)(P_in x_t)^T over unmasked tokens.
    Returns [B, k_out*k_in] float64, flat index o*k_in + i."""
    return _project(lib().oracle_project_factored, x, dy, p_in, p_out, mask)


def project_factored_layers(layers, mask=None) -> list:
    """project_factored for several layers of one batch, parallel over (layer, example).
    layers: list of (x, dy, p_in, p_out) of one dtype, shared B, T, k_in, k_out.
    Returns one [B, k_out*k_in] float64 array per layer."""
    n = len(layers)
    layers = [tuple(map(_c, L)) for L in layers]
    x0, _, pi0, po0 = layers[0]
    B, T, _ = x0.shape
    k_in, k_out = pi0.shape[0], po0.shape[0]
    code = _code(x0)
    for x, dy, pi, po in layers:
        assert all(_code(a) == code for a in (x, dy, pi, po))
        assert x.shape[:2] == (B, T) and dy.shape[:2] == (B, T)
        assert pi.shape == (k_in, x.shape[2]) and po.shape == (k_out, dy.shape[2])
    if mask is not None:
        mask = np.ascontiguousarray(mask.astype(np.uint8, copy=False))
        assert mask.shape == (B, T)
    gs = [np.zeros((B, k_out * k_in), dtype=np.float64) for _ in range(n)]
    ptrs = lambda arrs: (ctypes.c_void_p * n)(*[a.ctypes.data for a in arrs])
    ints = lambda v: (ctypes.c_int * n)(*v)
    rc = lib().oracle_project_factored_layers(
        n, ptrs([L[0] for L in layers]), ptrs([L[1] for L in layers]), code, B, T,
        ints([L[0].shape[2] for L in layers]), ints([L[1].shape[2] for L in layers]), _ptr(mask),
        ptrs([L[2] for L in layers]), ptrs([L[3] for L in layers]), k_in, k_out, ptrs(gs))
    _check(rc, "oracle_project_factored_layers")
    return gs


def project_dense(x, dy, p_in, p_out, mask=None) -> np.ndarray:
    """Eq. (4) then Eq. (5) left side: P_out (sum_t dy_t x_t^T) P_in^T.  Small inputs only."""
    return _project(lib().oracle_project_dense, x, dy, p_in, p_out, mask)


def cov_accumulate(g, S=None) -> np.ndarray:
    """S += sum_b g_b g_b^T (float64).  g: [B, D] (any oracle dtype)."""
    g = _c(g)
    B, D = g.shape
    if S is None:
        S = np.zeros((D, D), dtype=np.float64)
    assert S.dtype == np.float64 and S.shape == (D, D) and S.flags.c_contiguous
    rc = lib().oracle_cov_accumulate(_ptr(g), _code(g), D, B, D, _ptr(S))
    _check(rc, "oracle_cov_accumulate")
    return S


def precondition(S, N: int, damp_ratio: float, g_test):
    """(S/N + lambda I)^{-1} g_q for each row q, lambda = damp_ratio * tr(S/N) / D.
    damp_ratio < 0: identity.  Returns (out [Q, D] float64, lambda)."""
    S = np.ascontiguousarray(S, dtype=np.float64)
    g_test = _c(g_test)
    Q, D = g_test.shape
    assert S.shape == (D, D)
    out = np.zeros((Q, D), dtype=np.float64)
    lam = ctypes.c_double(0.0)
    rc = lib().oracle_precondition(_ptr(S), D, int(N), float(damp_ratio), _ptr(g_test),
                                   _code(g_test), D, Q, _ptr(out), D, ctypes.byref(lam))
    _check(rc, "oracle_precondition")
    return out, lam.value


def precondition_status(S, N: int, damp_ratio: float, g_test) -> int:
    """Status code of oracle_precondition (OK or ERR_NOT_PD) without raising."""
    S = np.ascontiguousarray(S, dtype=np.float64)
    g_test = _c(g_test)
    Q, D = g_test.shape
    out = np.zeros((Q, D), dtype=np.float64)
    return lib().oracle_precondition(_ptr(S), D, int(N), float(damp_ratio), _ptr(g_test),
                                     _code(g_test), D, Q, _ptr(out), D, None)


def scores(te, tr) -> np.ndarray:
    """s[q, j] = <te_q, tr_j> in float64.  te: [Q, D], tr: [N, D]."""
    te, tr = _c(te), _c(tr)
    Q, D = te.shape
    N = tr.shape[0]
    assert tr.shape[1] == D
    s = np.zeros((Q, N), dtype=np.float64)
    rc = lib().oracle_scores(_ptr(te), _code(te), D, Q, _ptr(tr), _code(tr), D, N, D, _ptr(s),
                             max(N, 1))
    _check(rc, "oracle_scores")
    return s


def topk(s, k: int, base: int = 0):
    """Top-k per row: largest values first, ties to the lower index; pads (-inf, -1).
    Returns (val [Q, k] float64, idx [Q, k] int64)."""
    s = np.ascontiguousarray(s, dtype=np.float64)
    Q, N = s.shape
    val = np.empty((Q, k), dtype=np.float64)
    idx = np.empty((Q, k), dtype=np.int64)
    rc = lib().oracle_topk(_ptr(s), max(N, 1), Q, N, int(base), int(k), _ptr(val), _ptr(idx))
    _check(rc, "oracle_topk")
    return val, idx


def self_influence(S, N: int, damp_ratio: float, g) -> np.ndarray:
    """self_j = g_j^T (S/N + lambda I)^{-1} g_j for one block (l-RelatIF's normaliser).
    damp_ratio < 0: identity (self = |g_j|^2).  Returns [rows] float64."""
    S = np.ascontiguousarray(S, dtype=np.float64)
    g = _c(g)
    rows, D = g.shape
    assert S.shape == (D, D)
    out = np.zeros(max(rows, 1), dtype=np.float64)
    rc = lib().oracle_self_influence(_ptr(S), D, int(N), float(damp_ratio), _ptr(g), _code(g), D, rows, _ptr(out))
    _check(rc, "oracle_self_influence")
    return out[:rows]


def self_influence_blocks(S_blocks, N: int, damp_ratio: float, g) -> np.ndarray:
    """Whole-model self-influence of a block-diagonal Hessian: the sum over column blocks."""
    nb, D, _ = np.shape(S_blocks)
    g = np.asarray(g)
    return sum(self_influence(S_blocks[l], N, damp_ratio, np.ascontiguousarray(g[:, l * D:(l + 1) * D]))
               for l in range(nb))


def normalise_scores(s, self_tr, self_te=None) -> np.ndarray:
    """l-RelatIF: s[q, j] / sqrt(self_tr[j]); cosine when self_te is given (also / sqrt(self_te[q]))."""
    s = np.array(s, dtype=np.float64, order="C")
    Q, N = s.shape
    tr = np.ascontiguousarray(self_tr, dtype=np.float64)
    te = None if self_te is None else np.ascontiguousarray(self_te, dtype=np.float64)
    rc = lib().oracle_normalise_scores(_ptr(s), max(N, 1), Q, N, None if te is None else _ptr(te), _ptr(tr))
    _check(rc, "oracle_normalise_scores")
    return s


def act_cov(a, mask=None, C=None) -> np.ndarray:
    """KFAC factor of one layer (Sec. 3.2): C += sum over unmasked tokens of a_t a_t^T.
    a: [B, T, n] (activations x for C_F, output gradients dy for C_B); returns [n, n] float64."""
    a = _c(a)
    B, T, n = a.shape
    if mask is not None:
        mask = np.ascontiguousarray(mask.astype(np.uint8, copy=False))
        assert mask.shape == (B, T)
    if C is None:
        C = np.zeros((n, n), dtype=np.float64)
    assert C.dtype == np.float64 and C.shape == (n, n) and C.flags.c_contiguous
    rc = lib().oracle_act_cov(_ptr(a), _code(a), B, T, n, _ptr(mask), _ptr(C))
    _check(rc, "oracle_act_cov")
    return C


def pca_topk(C, k: int):
    """PCA initialisation of a projection (Sec. 3.2): the top-k eigenvectors of the symmetric
    covariance C as the rows of P [k, n], by decreasing eigenvalue, each signed so that its entry
    of largest magnitude (the lowest index among equal magnitudes) is positive.  The
    eigendecomposition is numpy's float64 eigh.  Returns (P, eigenvalues [k])."""
    C = np.asarray(C, dtype=np.float64)
    n = C.shape[0]
    assert C.shape == (n, n) and 1 <= k <= n
    w, V = np.linalg.eigh(C)                 # ascending
    order = np.argsort(-w, kind="stable")[:k]
    P = V[:, order].T.copy()
    for r in range(k):
        i = int(np.argmax(np.abs(P[r])))     # first index of the largest magnitude
        if P[r, i] < 0:
            P[r] = -P[r]
    return P, w[order]


def num_threads() -> int:
    return int(lib().oracle_num_threads())
