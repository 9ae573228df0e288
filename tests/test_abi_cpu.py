"""The C-ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before touching the GPU.  CPU only: every call here
returns from host-side validation or is a pure size query."""
import ctypes
import os
import re

import pytest

import paper_2405_13954_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "logra.h")


def declared_symbols():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(logra_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(P.LIB_PATH):
        pytest.fail("libpaper_logra.so is not built (run __graft_entry__.build())")
    return P.lib()


def test_exports_every_declared_symbol(L):
    syms = declared_symbols()
    assert len(syms) >= 13
    for s in syms:
        assert hasattr(L, s), f"missing export {s}"
    assert set(syms) == set(P.EXPORTED)


def test_version(L):
    assert "gfx950" in P.logra_version()


def test_workspace_sizes(L):
    # chunk partials (one 64 x 16 fp32 block per side per 64-token tile at k <= 16, chunks of
    # 6144 columns at k <= 32), per-tile sums in 16 x 16 blocks ((16 KT)^2 floats a tile), the list
    # of non-empty tiles (+ its count), their 64-bit valid-token sets and every tile's set, each
    # rounded up to 256 bytes
    assert P.logra_project_ws_size(2, 100, 64, 48, 8, 12) == 2 * 2 * 2 * 64 * 16 * 4 + 4 * 256 * 4 + 3 * 256
    assert P.logra_project_ws_size(0, 100, 64, 48, 8, 8) == 0
    shapes = [(4096, 4096), (4096, 1024), (4096, 1024), (4096, 4096), (4096, 14336), (4096, 14336), (14336, 4096)]
    descs = (P.LayerDesc * 7)(*[P.LayerDesc(0, 0, 0, 0, 0, a, b) for a, b in shapes])
    # k = 64: chunks of up to 14336 columns -> 14 chunk blocks of 64 x 64 floats per tile
    want = 14 * 16 * 16 * 64 * 64 * 4 + 7 * 16 * 16 * 4096 * 4 + 1280 + 2 * 2048
    assert P.logra_project_layers_ws_size(descs, 7, 16, 1024, 64, 64) == want
    assert P.logra_precondition_ws_size(256, 224, 1024) >= 224 * 256 * 256 * 8
    assert P.logra_influence_ws_size(4, 10, 3, 0) == 256
    assert P.logra_influence_ws_size(4, 10, 3, 1) == 0
    # large chunks add per-query thresholds, counts and candidate lists
    # (8192 candidates of 4-byte value and 4-byte column)
    Q, N = 1024, 500_000
    cand = 2 * 4096 + 2 * 4 * Q * 8192
    assert P.logra_influence_ws_size(Q, N, 100, 0) == 4 * Q * N + cand
    assert P.logra_influence_ws_size(Q, N, 100, 1) == cand
    assert P.logra_influence_ws_size(Q, N, 0, 1) == 0


NULL = None


def proj(L, **kw):
    a = dict(x=NULL, dy=NULL, in_dtype=1, B=2, T=8, n_in=64, n_out=64, mask=NULL, p_in=NULL, p_out=NULL,
             k_in=8, k_out=8, g_out=NULL, g_dtype=0, g_ld=64, ws=NULL, ws_bytes=0, stream=NULL)
    a.update(kw)
    return L.logra_project_layer(*a.values())


def test_project_validation(L):
    assert proj(L, B=-1) == P.ERR_INVALID_ARG
    assert proj(L, n_in=0) == P.ERR_INVALID_ARG
    assert proj(L, n_in=60) == P.ERR_INVALID_ARG            # bf16 rows need multiples of 8
    assert proj(L, in_dtype=0, n_in=62) == P.ERR_INVALID_ARG  # fp32 rows need multiples of 4
    assert proj(L, in_dtype=7) == P.ERR_INVALID_ARG
    assert proj(L, k_in=129) == P.ERR_UNSUPPORTED
    assert proj(L, g_ld=63) == P.ERR_INVALID_ARG
    assert "g_ld" in P.logra_last_error()
    assert proj(L, B=0) == P.OK                              # no-op, no device access
    assert proj(L, T=0) == P.OK
    assert L.logra_project_layers(None, 1, 1, 2, 8, None, 8, 8, 0, 64, None, 0, None) == P.ERR_INVALID_ARG
    descs = (P.LayerDesc * 49)()
    assert L.logra_project_layers(descs, 49, 1, 2, 8, None, 8, 8, 0, 64, None, 0, None) == P.ERR_UNSUPPORTED


def test_cov_validation(L):
    assert L.logra_cov_accumulate(None, 1, 64, 4, 0, None, None) == P.ERR_INVALID_ARG
    assert L.logra_cov_accumulate(None, 1, 60, 4, 60, None, None) == P.ERR_INVALID_ARG   # bf16 needs D%8==0
    assert L.logra_cov_accumulate(None, 1, 32, 4, 64, None, None) == P.ERR_INVALID_ARG   # ld < D
    assert L.logra_cov_accumulate(None, 1, 64, 0, 64, None, None) == P.OK                # B = 0 no-op
    assert L.logra_cov_accumulate_blocks(None, 1, 512, 4, 256, 0, None, None) == P.ERR_INVALID_ARG
    f = L.logra_cov_accumulate_blocks_lower
    assert f(None, 1, 512, 4, 256, 0, None, None) == P.ERR_INVALID_ARG                 # n_blocks = 0
    assert f(None, 1, 508, 4, 254, 2, None, None) == P.ERR_INVALID_ARG                 # bf16 needs D%8==0
    assert f(None, 1, 256, 4, 256, 2, None, None) == P.ERR_INVALID_ARG                 # ld < D * n_blocks
    assert f(None, 7, 512, 4, 256, 2, None, None) == P.ERR_INVALID_ARG                 # bad dtype
    assert f(None, 1, 512, 0, 256, 2, None, None) == P.OK                              # B = 0 no-op


def test_precondition_validation(L):
    f = L.logra_precondition
    assert f(None, 8193, 4, 0.1, None, 0, 8193, 1, None, 0, 8193, None, 0, None) == P.ERR_UNSUPPORTED
    assert f(None, 64, 0, 0.1, None, 0, 64, 1, None, 0, 64, None, 0, None) == P.ERR_INVALID_ARG
    assert f(None, 64, 4, float("nan"), None, 0, 64, 1, None, 0, 64, None, 0, None) == P.ERR_INVALID_ARG
    assert f(None, 64, 4, 0.1, None, 0, 32, 1, None, 0, 64, None, 0, None) == P.ERR_INVALID_ARG
    assert f(None, 64, 4, -1.0, None, 0, 64, 0, None, 0, 64, None, 0, None) == P.OK     # identity, Q=0


def test_influence_validation(L):
    f = L.logra_influence_scores
    args = lambda **kw: [kw.get(k, v) for k, v in dict(
        te=None, tdt=1, ld_te=64, Q=2, tr=None, rdt=1, ld_tr=64, N=10, D=64, base=0, s=None, ld_s=10,
        topk=3, tv=None, ti=None, merge=0, ws=None, wsb=0, st=None).items()]
    assert f(*args(rdt=0)) == P.ERR_UNSUPPORTED
    assert f(*args(topk=1025)) == P.ERR_UNSUPPORTED
    assert f(*args(topk=0)) == P.ERR_INVALID_ARG          # nothing requested
    assert f(*args(D=60, ld_te=60, ld_tr=60)) == P.ERR_INVALID_ARG
    assert f(*args(merge=2)) == P.ERR_INVALID_ARG
    assert f(*args(base=-1)) == P.ERR_INVALID_ARG
    assert f(*args(Q=0)) == P.OK


def test_self_influence_ws_and_validation(L):
    # the preconditioner's workspace for Q = D (the identity solve) plus the
    # inverse factor's two bf16 halves, each [n_blocks][D rounded up to 256][D]
    assert P.logra_self_influence_ws_size(256, 224) == (P.logra_precondition_ws_size(256, 224, 256)
                                                        + 2 * 224 * 256 * 256 * 2)
    assert P.logra_self_influence_ws_size(40, 3) == (P.logra_precondition_ws_size(40, 3, 40)
                                                     + 2 * ((3 * 256 * 40 * 2 + 255) // 256 * 256))
    assert P.logra_self_influence_ws_size(0, 3) == 0
    f = L.logra_self_influence_blocks
    fake = ctypes.c_void_p(0x1000)    # never dereferenced: every case fails host validation first
    args = lambda **kw: [kw.get(k, v) for k, v in dict(
        S=None, D=64, nb=2, N=4, damp=0.1, g=None, gdt=1, ld=128, rows=4, so=fake, ro=None, ws=None, wsb=0,
        st=None).items()]
    assert f(*args(gdt=5)) == P.ERR_INVALID_ARG
    assert f(*args(D=0)) == P.ERR_INVALID_ARG
    assert f(*args(rows=-1)) == P.ERR_INVALID_ARG
    assert f(*args(D=8193, ld=8193 * 2)) == P.ERR_UNSUPPORTED
    assert f(*args(ld=127)) == P.ERR_INVALID_ARG
    assert f(*args(damp=float("nan"))) == P.ERR_INVALID_ARG
    assert f(*args(N=0)) == P.ERR_INVALID_ARG
    assert f(*args(so=None)) == P.ERR_INVALID_ARG          # nothing requested
    assert "nothing to compute" in P.logra_last_error()
    assert f(*args(D=60, ld=120)) == P.ERR_INVALID_ARG       # bf16 rows need multiples of 8
    assert f(*args(ld=1 << 22)) == P.ERR_UNSUPPORTED
    assert f(*args(rows=0, so=None)) == P.OK                # no rows: a no-op, no device access


def test_scaled_influence_validation(L):
    f = L.logra_influence_scores_scaled
    args = lambda **kw: [kw.get(k, v) for k, v in dict(
        te=None, tdt=1, ld_te=64, Q=2, tr=None, rdt=1, ld_tr=64, N=10, D=64, base=0, rs=None, cs=None, s=None,
        ld_s=10, topk=3, tv=None, ti=None, merge=0, ws=None, wsb=0, st=None).items()]
    assert f(*args(rdt=0)) == P.ERR_UNSUPPORTED
    assert f(*args(topk=1025)) == P.ERR_UNSUPPORTED
    assert f(*args(topk=0)) == P.ERR_INVALID_ARG
    assert f(*args(Q=0)) == P.OK


def test_pca_entry_points_validation(L):
    # activation covariance: the slab list (one int and one 32-bit token map per
    # 32-token slab) and its count
    assert P.logra_act_cov_ws_size(8, 2048) == 2 * (8 * 64 * 4) + 256
    assert P.logra_act_cov_ws_size(0, 16) == 0
    f = L.logra_act_cov_accumulate
    fake = ctypes.c_void_p(0x1000)
    assert f(None, 5, 2, 4, 64, None, fake, None, 0, None) == P.ERR_INVALID_ARG     # dtype
    assert f(None, 1, 2, 4, 60, None, fake, None, 0, None) == P.ERR_INVALID_ARG     # bf16 n % 8
    assert f(None, 1, -1, 4, 64, None, fake, None, 0, None) == P.ERR_INVALID_ARG
    assert f(None, 1, 0, 4, 64, None, fake, None, 0, None) == P.OK                  # no tokens: a no-op
    # the grouped form: descriptor limits, per-factor sizes, overlapping outputs
    grp = L.logra_act_cov_accumulate_group
    D = P.ActCovDesc
    two = (D * 2)(D(0x1000, 0x100000, 64), D(0x1000, 0x200000, 64))
    assert grp(None, 1, 1, 2, 4, None, None, 0, None) == P.ERR_INVALID_ARG          # no descriptors
    assert grp(two, 0, 1, 2, 4, None, None, 0, None) == P.ERR_INVALID_ARG
    many = (D * (P.MAX_ACT_COV_GROUP + 1))()
    assert grp(many, P.MAX_ACT_COV_GROUP + 1, 1, 2, 4, None, None, 0, None) == P.ERR_UNSUPPORTED
    assert grp(two, 2, 5, 2, 4, None, None, 0, None) == P.ERR_INVALID_ARG           # dtype
    bad = (D * 2)(D(0x1000, 0x100000, 64), D(0x1000, 0x200000, 60))
    assert grp(bad, 2, 1, 2, 4, None, None, 0, None) == P.ERR_INVALID_ARG           # bf16 n % 8
    assert "factor 1" in P.logra_last_error()
    grp(bad, 2, 0, 2, 4, None, None, 0, None)                                          # fp32: any n
    assert "multiple of 8" not in P.logra_last_error()
    big = (D * 1)(D(0x1000, 0x100000, (1 << 20) + 8))
    assert grp(big, 1, 1, 2, 4, None, None, 0, None) == P.ERR_UNSUPPORTED
    assert grp(two, 2, 1, 0, 4, None, None, 0, None) == P.OK                          # no tokens: a no-op
    # C of factor 1 starts inside factor 0's 64 x 64 floats (16 KB): rejected before any launch
    clash = (D * 2)(D(0x1000, 0x100000, 64), D(0x1000, 0x100000 + 16380, 64))
    assert grp(clash, 2, 1, 2, 4, None, None, 0, None) == P.ERR_INVALID_ARG
    assert "overlap" in P.logra_last_error()
    # back to back is not an overlap (the call then fails on the pointers, which are not device memory)
    touch = (D * 2)(D(0x1000, 0x100000, 64), D(0x1000, 0x100000 + 16384, 64))
    assert grp(touch, 2, 1, 2, 4, None, None, 0, None) == P.ERR_INVALID_ARG
    assert "overlap" not in P.logra_last_error()
    # PCA: k limits, iterations, output stride
    assert P.logra_pca_ws_size(100, 65) == 0 and P.logra_pca_ws_size(10, 11) == 0
    assert P.logra_pca_ws_size(4096, 16) > 2 * 4096 * 32 * 4
    g = L.logra_pca_topk
    assert g(fake, 100, 0, 30, fake, 0, 100, None, None, 0, None) == P.ERR_INVALID_ARG
    assert g(fake, 100, 65, 30, fake, 0, 100, None, None, 0, None) == P.ERR_UNSUPPORTED
    assert g(fake, 10, 11, 30, fake, 0, 10, None, None, 0, None) == P.ERR_INVALID_ARG
    assert g(fake, 100, 8, 0, fake, 0, 100, None, None, 0, None) == P.ERR_INVALID_ARG
    assert g(fake, 100, 8, 30, fake, 0, 99, None, None, 0, None) == P.ERR_INVALID_ARG


def test_influence_stream_ws_and_validation(L):
    # two staging buffers of chunk_rows x D plus one chunk's scoring workspace
    assert P.logra_influence_stream_ws_size(16, 1000, 64, P.BF16, 10) == (
        2 * ((1000 * 64 * 2 + 255) // 256 * 256) + P.logra_influence_ws_size(16, 1000, 10, 0))
    assert P.logra_influence_stream_ws_size(16, 0, 64, P.BF16, 10) == 0
    f = L.logra_influence_stream
    args = lambda **kw: [kw.get(k, v) for k, v in dict(
        te=None, tdt=1, ld_te=64, Q=2, tr=None, rdt=1, ld_tr=64, N=10, D=64, chunk=4, topk=3, tv=None,
        ti=None, ws=None, wsb=0, st=None, cst=None).items()]
    assert f(*args(rdt=0)) == P.ERR_UNSUPPORTED
    assert f(*args(topk=0)) == P.ERR_INVALID_ARG
    assert f(*args(topk=1025)) == P.ERR_UNSUPPORTED
    assert f(*args(chunk=0)) == P.ERR_INVALID_ARG
    assert f(*args(ld_tr=32)) == P.ERR_INVALID_ARG
    assert f(*args(D=60, ld_te=60, ld_tr=60)) == P.ERR_INVALID_ARG
    assert f(*args(Q=0)) == P.OK


def test_offload_rows_validation(L):
    f = L.logra_offload_rows
    args = lambda **kw: [kw.get(k, v) for k, v in dict(
        src=None, ld_src=64, dst=None, ld_dst=64, rows=4, row_bytes=64, st=None, cst=None, done=None).items()]
    assert f(*args(rows=-1)) == P.ERR_INVALID_ARG
    assert f(*args(row_bytes=0)) == P.ERR_INVALID_ARG
    assert f(*args(ld_src=32)) == P.ERR_INVALID_ARG
    assert f(*args(ld_dst=63)) == P.ERR_INVALID_ARG
    assert f(*args(rows=0)) == P.OK                       # nothing to copy: no pointer is looked at
    assert f(*args()) == P.ERR_INVALID_ARG                 # NULL src


def test_f64_statistics_validation(L):
    """The float64 statistics path: fp64 S, fp64 preconditioned gradients and
    float64-accumulated scores are accepted where documented, and refused
    elsewhere."""
    assert proj(L, g_dtype=P.F64) == P.ERR_INVALID_ARG        # projections store fp32 or bf16
    assert proj(L, in_dtype=P.F64) == P.ERR_INVALID_ARG
    c = L.logra_cov_accumulate_f64
    assert c(None, P.BF16, 64, 4, 64, 1, None, None) == P.ERR_INVALID_ARG   # fp32 / fp64 rows only
    assert c(None, P.F32, 100, 4, 64, 2, None, None) == P.ERR_INVALID_ARG   # ld < D * n_blocks
    assert c(None, P.F32, 64, 4, 64, 0, None, None) == P.ERR_INVALID_ARG
    assert c(None, P.F64, 64 * 65536, 4, 64, 65536, None, None) == P.ERR_UNSUPPORTED
    assert c(None, P.F64, 64, 0, 64, 1, None, None) == P.OK                 # B = 0: a no-op
    assert L.logra_cov_accumulate(None, P.F64, 64, 4, 64, None, None) == P.ERR_INVALID_ARG  # fp32 S
    p = L.logra_precondition_f64
    assert p(None, 8193, 1, 4, 0.1, None, P.F32, 8193, 1, None, P.F64, 8193, None, 0, None) == P.ERR_UNSUPPORTED
    assert p(None, 64, 1, 4, 0.1, None, 3, 64, 1, None, P.F64, 64, None, 0, None) == P.ERR_INVALID_ARG
    assert p(None, 64, 1, 0, 0.1, None, P.F32, 64, 1, None, P.F64, 64, None, 0, None) == P.ERR_INVALID_ARG
    assert p(None, 64, 2, 4, 0.1, None, P.F32, 100, 1, None, P.F64, 128, None, 0, None) == P.ERR_INVALID_ARG
    assert p(None, 64, 1, 4, -1.0, None, P.F64, 64, 0, None, P.F64, 64, None, 0, None) == P.OK
    f = L.logra_influence_scores
    args = lambda **kw: [kw.get(k, v) for k, v in dict(
        te=None, tdt=P.F64, ld_te=64, Q=2, tr=None, rdt=P.F32, ld_tr=64, N=10, D=64, base=0, s=None, ld_s=10,
        topk=3, tv=None, ti=None, merge=0, ws=None, wsb=0, st=None).items()]
    assert f(*args(rdt=P.BF16)) == P.ERR_UNSUPPORTED           # bf16 pairs only with bf16
    assert f(*args(tdt=P.BF16, rdt=P.F64)) == P.ERR_UNSUPPORTED
    assert f(*args(tdt=3)) == P.ERR_INVALID_ARG
    assert f(*args(Q=70000)) == P.ERR_UNSUPPORTED
    assert f(*args(Q=0)) == P.OK
    assert f(*args()) == P.ERR_INVALID_ARG                     # passes the dtype checks; NULL top-k buffers
    assert "topk_val" in P.logra_last_error()


def test_peaks_library_exports_and_validation():
    """The measured-ceiling library (include/logra_peaks.h) loads, exports what
    its header declares, and refuses bad arguments before any launch."""
    path = os.path.join(os.path.dirname(P.LIB_PATH), "libpaper_logra_peaks.so")
    if not os.path.exists(path):
        pytest.fail("libpaper_logra_peaks.so is not built (run __graft_entry__.build())")
    src = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "logra_peaks.h")).read(), flags=re.S)
    syms = sorted(set(re.findall(r"\b(logra_[a-z_0-9]+)\s*\(", src)))
    K = ctypes.CDLL(path)
    assert syms == ["logra_peak_hbm_read", "logra_peak_mfma_bf16", "logra_peak_mfma_bf16_data",
                    "logra_peak_wall_clock_khz"]
    for s in syms:
        assert hasattr(K, s)
    K.logra_peak_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p]
    K.logra_peak_hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                      ctypes.c_void_p]
    fake = ctypes.c_void_p(0x1000)
    assert K.logra_peak_mfma_bf16(0, 10, fake, None, None) == -1
    assert K.logra_peak_mfma_bf16(4, 10, None, None, None) == -1
    K.logra_peak_mfma_bf16_data.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p]
    ops = ctypes.c_void_p(0x2000)
    assert K.logra_peak_mfma_bf16_data(4, 12, ops, fake, None, None) == -1             # not a multiple of 8
    assert K.logra_peak_mfma_bf16_data(4, 16, None, fake, None, None) == -1
    assert K.logra_peak_mfma_bf16_data(4, 16, ctypes.c_void_p(0x2008), fake, None, None) == -1   # unaligned
    assert K.logra_peak_mfma_bf16_data(0, 16, ops, fake, None, None) == -1
    big = ctypes.c_void_p(0x100000)
    assert K.logra_peak_hbm_read(big, 1000, 4, 0, fake, None) == -1      # not a multiple of 1 KB
    assert K.logra_peak_hbm_read(None, 1024, 4, 0, fake, None) == -1
    assert K.logra_peak_hbm_read(big, 1024, 4, 3, fake, None) == -1      # no such method
