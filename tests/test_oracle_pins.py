"""Pins of the float64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a hand-worked
example, an identity the paper states (Eq. (5), Lemma 1, the trace form of the
mean eigenvalue), a special case that reduces to a library routine, or an
invariant (symmetry, PSD, rank, additivity, masking).  A plausible slip in the
oracle -- a dropped term, a wrong sign, a transposed operand or index -- fails
at least one of them.  CPU only.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    den = max(np.max(np.abs(b)), 1e-300)
    return float(np.max(np.abs(a - b)) / den)


def _asym(seed=0, dtype="f32", B=3, T=7, n_in=48, n_out=80, k_in=4, k_out=12, ragged=True):
    g = W.rng(seed, 99)
    d = W.layer_inputs(seed, 0, B, T, n_in, n_out, k_in, k_out, 1.0, 0.5, dtype,
                       lens=(g.integers(0, T + 1, size=B) if ragged else None))
    if ragged:
        d["mask"][0, :] = 0          # one fully masked example
        d["mask"][-1, :] = 1         # one full example
    return d


def _f64(a):
    a = np.asarray(a)
    return W.bf16_bits_to_f32(a).astype(np.float64) if a.dtype == np.uint16 else a.astype(np.float64)


# --------------------------------------------------------------------------
# Golden hand-worked examples
# --------------------------------------------------------------------------
def test_golden_projection_2x2():
    e = json.load(open(GOLD))["logra_projection_2x2"]
    conv = lambda v: np.array([[float(z) for z in r] for r in v], dtype=np.float32)
    x = conv(e["x"])[None]
    dy = conv(e["dy"])[None]
    mask = np.array([e["mask"]], dtype=np.uint8)
    p_in, p_out = conv(e["p_in"]), conv(e["p_out"])
    want = np.array(e["G_flat_out_major"], dtype=np.float64)
    got = oracle.project_factored(x, dy, p_in, p_out, mask)[0]
    assert np.array_equal(got, want)
    got_d = oracle.project_dense(x, dy, p_in, p_out, mask)[0]
    assert np.array_equal(got_d, want)


def test_golden_lemma1_2x2():
    e = json.load(open(GOLD))["lemma1_2x2"]
    S = np.array(e["S"], dtype=np.float64)
    g_te = np.array([e["g_te"]], dtype=np.float64)
    g_tr = np.array([e["g_tr"]], dtype=np.float64)
    pre, lam = oracle.precondition(S, e["N"], e["damp_ratio"], g_te)
    assert lam == e["lambda"]
    assert np.allclose(pre[0], e["preconditioned_te"], rtol=0, atol=1e-15)
    s = oracle.scores(pre, g_tr)
    assert abs(s[0, 0] - e["score"]) < 1e-15


def test_golden_cov_2x3():
    e = json.load(open(GOLD))["cov_2x3"]
    S = oracle.cov_accumulate(np.array(e["g"], dtype=np.float64))
    assert np.array_equal(S, np.array(e["S"], dtype=np.float64))


# --------------------------------------------------------------------------
# P1: Eq. (5) is an exact identity -- factored == dense == explicit Kronecker
# --------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_eq5_factored_dense_kronecker(dtype):
    d = _asym(1, dtype)
    gf = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], d["mask"])
    gd = oracle.project_dense(d["x"], d["dy"], d["p_in"], d["p_out"], d["mask"])
    x, dy, pi, po = map(_f64, (d["x"], d["dy"], d["p_in"], d["p_out"]))
    k_in, k_out = pi.shape[0], po.shape[0]
    Pk = np.kron(pi, po)                      # P = P_i (x) P_o, Sec. 3.1
    B, T = d["mask"].shape
    for b in range(B):
        # Eq. (4): vec(DW) = sum_t x_t (x) Dx_t  (column-major vec of DW)
        vec_dw = np.zeros(x.shape[2] * dy.shape[2])
        for t in range(T):
            if d["mask"][b, t]:
                vec_dw += np.kron(x[b, t], dy[b, t])
        vec_g = Pk @ vec_dw                   # column-major: vec_g[i*k_out + o] = G[o, i]
        want = vec_g.reshape(k_in, k_out).T.reshape(-1)   # -> flat[o*k_in + i]
        scale = max(np.abs(want).max(), 1e-300)
        assert np.abs(gf[b] - want).max() / scale < 1e-12, b
        assert np.abs(gd[b] - want).max() / scale < 1e-12, b
    assert np.all(gf[0] == 0.0)               # fully masked example


def test_eq5_layout_is_out_major():
    """A transposed [k_in][k_out] layout would fail here: k_in != k_out, one nonzero."""
    x = np.zeros((1, 1, 8), np.float32); x[0, 0, 3] = 1.0
    dy = np.zeros((1, 1, 16), np.float32); dy[0, 0, 5] = 1.0
    p_in = np.zeros((2, 8), np.float32); p_in[1, 3] = 1.0      # x' = e_1 (k_in = 2)
    p_out = np.zeros((3, 16), np.float32); p_out[2, 5] = 1.0   # dy' = e_2 (k_out = 3)
    g = oracle.project_factored(x, dy, p_in, p_out)[0]
    want = np.zeros(6); want[2 * 2 + 1] = 1.0                  # flat[o*k_in + i], o=2, i=1
    assert np.array_equal(g, want)


# --------------------------------------------------------------------------
# P2: P = I reduces to the textbook per-example gradient sum_t dy_t x_t^T
# --------------------------------------------------------------------------
def test_identity_projection_gives_full_gradient():
    g = W.rng(5)
    B, T, n_in, n_out = 2, 5, 6, 4
    x = g.integers(-3, 4, size=(B, T, n_in)).astype(np.float32)
    dy = g.integers(-3, 4, size=(B, T, n_out)).astype(np.float32)
    mask = np.ones((B, T), np.uint8); mask[1, 3:] = 0
    G = oracle.project_factored(x, dy, np.eye(n_in, dtype=np.float32),
                                np.eye(n_out, dtype=np.float32), mask)
    for b in range(B):
        dw = np.einsum("ta,tc->ac", dy[b][mask[b] == 1].astype(np.float64),
                       x[b][mask[b] == 1].astype(np.float64))
        assert np.array_equal(G[b].reshape(n_out, n_in), dw)
    # coordinate-selection P returns the matching sub-block of DW
    rows_in, rows_out = [4, 1], [3, 0, 2]
    Gs = oracle.project_factored(x, dy, np.eye(n_in, dtype=np.float32)[rows_in],
                                 np.eye(n_out, dtype=np.float32)[rows_out], mask)
    for b in range(B):
        assert np.array_equal(Gs[b].reshape(3, 2), G[b].reshape(n_out, n_in)[np.ix_(rows_out, rows_in)])


# --------------------------------------------------------------------------
# P3: masking
# --------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mask_equals_deletion_and_ignores_nonfinite(dtype):
    d = _asym(2, dtype)
    m = d["mask"]
    base = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], m)
    # poison masked slots with NaN / Inf: result must be bitwise identical
    x, dy = d["x"].copy(), d["dy"].copy()
    if dtype == "f32":
        x[m == 0] = np.nan
        dy[m == 0] = np.inf
    else:
        x[m == 0] = 0x7FC0    # bf16 NaN
        dy[m == 0] = 0xFF80   # bf16 -Inf
    pois = oracle.project_factored(x, dy, d["p_in"], d["p_out"], m)
    assert np.array_equal(base, pois)
    assert np.all(np.isfinite(pois))
    # masked tokens == tokens deleted
    for b in range(m.shape[0]):
        keep = m[b] == 1
        one = oracle.project_factored(d["x"][b][keep][None], d["dy"][b][keep][None],
                                      d["p_in"], d["p_out"])
        assert np.array_equal(one[0], base[b])


def test_all_masked_and_empty():
    d = _asym(3)
    z = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], np.zeros_like(d["mask"]))
    assert np.all(z == 0.0)
    e = oracle.project_factored(d["x"][:0], d["dy"][:0], d["p_in"], d["p_out"], d["mask"][:0])
    assert e.shape == (0, d["p_in"].shape[0] * d["p_out"].shape[0])


# --------------------------------------------------------------------------
# P4: bilinearity and additivity over token subsets (split-T invariance)
# --------------------------------------------------------------------------
def test_scaling_and_additivity():
    d = _asym(4)
    m = d["mask"]
    G = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], m)
    G2 = oracle.project_factored(d["x"], d["dy"] * np.float32(4.0), d["p_in"], d["p_out"], m)
    assert np.array_equal(G2, 4.0 * G)
    Gx = oracle.project_factored(d["x"] * np.float32(-0.5), d["dy"], d["p_in"], d["p_out"], m)
    assert np.array_equal(Gx, -0.5 * G)
    T = m.shape[1]
    first = m.copy(); first[:, T // 2:] = 0
    second = m.copy(); second[:, :T // 2] = 0
    Ga = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], first)
    Gb = oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], second)
    assert _rel(Ga + Gb, G) < 1e-13


# --------------------------------------------------------------------------
# P5: covariance (Assumption 1): symmetric, PSD, rank <= N, trace, N=1, chunking
# --------------------------------------------------------------------------
def test_covariance_invariants():
    g = W.rng(6)
    N, D = 5, 24
    G = g.standard_normal((N, D))
    S = oracle.cov_accumulate(G)
    assert np.array_equal(S, S.T)
    ev = np.linalg.eigvalsh(S)
    assert ev.min() >= -1e-12 * np.trace(S)
    assert np.linalg.matrix_rank(S, tol=1e-9 * ev.max()) == N
    assert abs(np.trace(S) - sum(float(r @ r) for r in G)) < 1e-12 * np.trace(S)
    # N = 1 is the outer product, exactly (integer entries)
    gi = g.integers(-5, 6, size=(1, 7)).astype(np.float32)
    assert np.array_equal(oracle.cov_accumulate(gi), np.outer(gi[0], gi[0]).astype(np.float64))
    # chunked accumulation equals one call (integer entries: exact)
    Gi = g.integers(-4, 5, size=(9, 11)).astype(np.float32)
    one = oracle.cov_accumulate(Gi)
    parts = oracle.cov_accumulate(Gi[:4])
    oracle.cov_accumulate(Gi[4:], parts)
    assert np.array_equal(one, parts)


def test_covariance_bf16_input_and_stride():
    g = W.rng(7)
    Gf = g.standard_normal((6, 16)).astype(np.float32)
    Gb = W.f32_to_bf16_bits(Gf)
    S = oracle.cov_accumulate(Gb)
    Gw = W.bf16_bits_to_f32(Gb).astype(np.float64)
    # the widened bf16 values enter exactly: compare with the same data given as fp64
    assert _rel(S, oracle.cov_accumulate(Gw)) == 0.0


# --------------------------------------------------------------------------
# P6: damping lambda = r * mean(eigenvalues) = r * tr(C) / D  (App. C)
# --------------------------------------------------------------------------
def test_damping_is_mean_eigenvalue():
    g = W.rng(8)
    N, D = 7, 20
    G = g.standard_normal((N, D))
    S = oracle.cov_accumulate(G)
    for r in (0.1, 1e-3, 2.0):
        _, lam = oracle.precondition(S, N, r, G[:1])
        want = r * np.mean(np.linalg.eigvalsh(S / N))
        assert abs(lam - want) < 1e-12 * abs(want)


# --------------------------------------------------------------------------
# P7: preconditioning -- residual and the eigen-form of Lemma 1
# --------------------------------------------------------------------------
def test_precondition_residual_and_lemma1():
    g = W.rng(9)
    N, D, Q = 6, 16, 3              # rank-deficient covariance: damping matters
    G = g.standard_normal((N, D))
    S = oracle.cov_accumulate(G)
    C = S / N
    g_te = g.standard_normal((Q, D))
    g_tr = g.standard_normal((4, D))
    r = 0.1
    pre, lam = oracle.precondition(S, N, r, g_te)
    res = (C + lam * np.eye(D)) @ pre.T - g_te.T
    kappa = np.linalg.cond(C + lam * np.eye(D))
    assert np.abs(res).max() <= 1e-12 * kappa * np.abs(g_te).max()
    s = oracle.scores(pre, g_tr)
    # Lemma 1 (App. D proof): g_te^T Q (Lambda + lambda I)^{-1} Q^T g_tr
    ev, Qm = np.linalg.eigh(C)
    want = (g_te @ Qm) @ np.diag(1.0 / (ev + lam)) @ (g_tr @ Qm).T
    assert _rel(s, want) < 1e-10
    # and the sum form sum_i lambda_i/(lambda_i+lambda) c_tr,i c_te,i for gradients
    # in the span of the positive eigenvalues (the covariance's own samples)
    pos = ev > 1e-10 * ev.max()
    c_te = (G[:2] @ Qm[:, pos]) / np.sqrt(ev[pos])
    c_tr = (G[2:5] @ Qm[:, pos]) / np.sqrt(ev[pos])
    lemma = (c_te * (ev[pos] / (ev[pos] + lam))) @ c_tr.T
    pre2, _ = oracle.precondition(S, N, r, G[:2])
    assert _rel(oracle.scores(pre2, G[2:5]), lemma) < 1e-10


def test_precondition_identity_and_not_pd():
    g = W.rng(10)
    gt = g.standard_normal((3, 5)).astype(np.float32)
    out, _ = oracle.precondition(np.zeros((5, 5)), 1, -1.0, gt)
    assert np.array_equal(out, gt.astype(np.float64))
    # rank-deficient S with zero damping: the second pivot is exactly zero
    S = oracle.cov_accumulate(np.array([[1.0, 2.0]]))
    assert oracle.precondition_status(S, 1, 0.0, np.ones((1, 2))) == oracle.ERR_NOT_PD
    # a negative diagonal entry is not positive definite either
    S2 = np.array([[-1.0, 0.0], [0.0, 1.0]])
    assert oracle.precondition_status(S2, 1, 0.0, np.ones((1, 2))) == oracle.ERR_NOT_PD
    # small positive damping makes it definite
    assert oracle.precondition_status(S, 1, 1e-3, np.ones((1, 2))) == oracle.OK


# --------------------------------------------------------------------------
# Self-influence and normalised scores (l-RelatIF, Sec. 4.2)
# --------------------------------------------------------------------------
def test_self_influence_eigen_form_and_identity():
    g = W.rng(15)
    N, D = 5, 12                    # rank-deficient covariance: damping matters
    G = g.standard_normal((N, D))
    S = oracle.cov_accumulate(G)
    rows = g.standard_normal((6, D)).astype(np.float32)
    r = 0.1
    got = oracle.self_influence(S, N, r, rows)
    # eigen-form of g^T (C + lambda I)^{-1} g with an independent eigensolver
    C = S / N
    lam = r * np.trace(C) / D
    ev, Qm = np.linalg.eigh(C)
    c = rows.astype(np.float64) @ Qm
    want = (c * c / (ev + lam)).sum(axis=1)
    assert _rel(got, want) < 1e-10
    assert np.all(got > 0)
    # identity preconditioner: the squared norm
    ident = oracle.self_influence(np.zeros((D, D)), 1, -1.0, rows)
    assert np.allclose(ident, (rows.astype(np.float64) ** 2).sum(axis=1), rtol=1e-14, atol=0)
    # quadratic in g
    assert _rel(oracle.self_influence(S, N, r, 3 * rows.astype(np.float64)), 9 * got) < 1e-12


def test_normalised_scores_cosine_and_outlier_invariance():
    g = W.rng(16)
    N, D = 9, 10
    G = g.standard_normal((N, D))
    S = oracle.cov_accumulate(G)
    r = 0.05
    tr = g.standard_normal((7, D))
    te = g.standard_normal((4, D))
    pre, _ = oracle.precondition(S, N, r, te)
    s_tr = oracle.self_influence(S, N, r, tr)
    s_te = oracle.self_influence(S, N, r, te)
    cos = oracle.normalise_scores(oracle.scores(pre, tr), s_tr, s_te)
    assert np.abs(cos).max() <= 1.0 + 1e-12                     # Cauchy-Schwarz in the inverse metric
    pre_tr, _ = oracle.precondition(S, N, r, tr)
    self_cos = oracle.normalise_scores(oracle.scores(pre_tr, tr), s_tr, s_tr)
    assert np.allclose(np.diag(self_cos), 1.0, rtol=0, atol=1e-12)   # a gradient with itself
    # l-RelatIF: scaling a train gradient by a > 0 leaves its scores unchanged
    rel = oracle.normalise_scores(oracle.scores(pre, tr), s_tr)
    tr2 = tr.copy()
    tr2[3] *= 40.0
    rel2 = oracle.normalise_scores(oracle.scores(pre, tr2), oracle.self_influence(S, N, r, tr2))
    assert _rel(rel2, rel) < 1e-12
    # and it is the raw score over the square root of the self-influence
    assert _rel(rel, oracle.scores(pre, tr) / np.sqrt(s_tr)[None, :]) < 1e-14
    # a zero gradient normalises to zero scores
    z = oracle.normalise_scores(np.zeros((2, 3)), np.array([0.0, 1.0, 4.0]))
    assert np.all(z == 0)


# --------------------------------------------------------------------------
# P8: scores -- identity preconditioner is a plain dot product; limits
# --------------------------------------------------------------------------
def test_scores_dot_product_and_limits():
    g = W.rng(11)
    te = g.standard_normal((3, 40)).astype(np.float32)
    tr = g.standard_normal((9, 40)).astype(np.float32)
    pre, _ = oracle.precondition(np.zeros((40, 40)), 1, -1.0, te)
    s = oracle.scores(pre, tr)
    assert _rel(s, te.astype(np.float64) @ tr.astype(np.float64).T) < 1e-14
    # bf16 inputs widen exactly
    tb = W.f32_to_bf16_bits(tr)
    assert _rel(oracle.scores(te, tb), te.astype(np.float64) @ W.bf16_bits_to_f32(tb).astype(np.float64).T) < 1e-14
    # symmetric in the two sides when both are preconditioned the same way
    G = g.standard_normal((10, 12))
    S = oracle.cov_accumulate(G)
    a, b = G[:1], G[1:2]
    pa, _ = oracle.precondition(S, 10, 0.1, a)
    pb, _ = oracle.precondition(S, 10, 0.1, b)
    assert abs(oracle.scores(pa, b)[0, 0] - oracle.scores(pb, a)[0, 0]) < 1e-12 * np.abs(pa).max() * np.abs(b).max() * 12
    # self-influence is positive
    assert oracle.scores(pa, a)[0, 0] > 0
    # heavy damping: lambda * s -> g_te . g_tr
    big, lam = oracle.precondition(S, 10, 1e8, a)
    assert abs(lam * oracle.scores(big, b)[0, 0] - float(a[0] @ b[0])) < 1e-6 * abs(float(a[0] @ b[0])) + 1e-9


# --------------------------------------------------------------------------
# P9: top-k -- equals a full stable sort with ties to the lower index
# --------------------------------------------------------------------------
def test_topk_matches_full_sort_with_ties():
    g = W.rng(12)
    Q, N, k = 4, 300, 17
    s = np.round(g.standard_normal((Q, N)) * 4) / 4        # many exact ties
    val, idx = oracle.topk(s, k, base=1000)
    for q in range(Q):
        order = np.lexsort((np.arange(N), -s[q]))[:k]      # value desc, then index asc
        assert np.array_equal(idx[q], order + 1000)
        assert np.array_equal(val[q], s[q, order])


def test_topk_padding_and_chunk_merge():
    g = W.rng(13)
    s = g.standard_normal((2, 3))
    val, idx = oracle.topk(s, 5)
    assert np.all(idx[:, 3:] == -1) and np.all(np.isneginf(val[:, 3:]))
    # top-k over the whole row == top-k of the union of per-chunk top-k lists
    s = np.round(g.standard_normal((3, 500)) * 3) / 3
    full_v, full_i = oracle.topk(s, 10)
    cand_v, cand_i = [], []
    for c0 in range(0, 500, 128):
        v, i = oracle.topk(s[:, c0:c0 + 128], 10, base=c0)
        cand_v.append(v); cand_i.append(i)
    cv, ci = np.concatenate(cand_v, 1), np.concatenate(cand_i, 1)
    for q in range(3):
        ok = ci[q] >= 0
        order = np.lexsort((ci[q][ok], -cv[q][ok]))[:10]
        assert np.array_equal(ci[q][ok][order], full_i[q])


# --------------------------------------------------------------------------
# KFAC factors and the PCA initialisation of the projections (Sec. 3.2)
# --------------------------------------------------------------------------
def test_golden_kfac_pca_2x2():
    e = json.load(open(GOLD))["kfac_pca_2x2"]
    a = np.array([[float(v) for v in row] for row in e["a"]])[None]
    C = oracle.act_cov(a, np.array([e["mask"]], np.uint8))
    assert np.array_equal(C, np.array(e["C_F"], np.float64))
    P, w = oracle.pca_topk(C, 2)
    assert np.allclose(w, e["eigvals"], rtol=0, atol=1e-13)
    assert np.allclose(P, e["P_top2"], rtol=0, atol=1e-15)
    H = np.kron(C, np.array(e["C_B"], np.float64))
    Pk, wk = oracle.pca_topk(H, 1)
    assert abs(wk[0] - e["kfac_top_eigval"]) < 1e-12
    assert np.allclose(Pk[0], e["kfac_top_eigvec"], rtol=0, atol=1e-15)


def test_act_cov_mask_is_deletion_and_invariants():
    g = W.rng(17)
    B, T, n = 3, 9, 12
    a = g.standard_normal((B, T, n))
    mask = (g.random((B, T)) < 0.6).astype(np.uint8)
    mask[0] = 0                                   # a fully masked example
    a_nan = a.copy()
    a_nan[mask == 0] = np.nan                     # masked slots are never read
    C = oracle.act_cov(a_nan, mask)
    kept = a[mask > 0]                            # the valid tokens, in order
    assert np.array_equal(C, oracle.act_cov(kept[None]))
    assert np.array_equal(C, C.T)
    assert abs(np.trace(C) - np.sum(kept ** 2)) <= 1e-12 * np.trace(C)
    ev = np.linalg.eigvalsh(C)
    assert ev.min() >= -1e-12 * ev.max()
    assert np.linalg.matrix_rank(oracle.act_cov(kept[:5][None])) == 5    # rank = tokens < n
    # one token gives its outer product exactly; accumulating two halves gives the whole
    assert np.array_equal(oracle.act_cov(kept[:1][None]), np.outer(kept[0], kept[0]))
    half = oracle.act_cov(a_nan[:2], mask[:2])
    both = oracle.act_cov(a_nan[2:], mask[2:], C=half.copy())
    assert _rel(both, C) < 1e-14
    # bf16 inputs are widened exactly
    ab = W.f32_to_bf16_bits(a.astype(np.float32))
    assert np.array_equal(oracle.act_cov(ab, mask), oracle.act_cov(_f64(ab), mask))


def test_pca_topk_eigen_properties():
    n, k = 40, 7
    C = W.spd_matrix(18, n, n).astype(np.float64)
    P, w = oracle.pca_topk(C, k)
    assert np.all(np.diff(w) <= 0)                                  # descending
    assert _rel(C @ P.T, P.T * w) < 1e-12                          # eigenpairs
    assert _rel(P @ P.T, np.eye(k)) < 1e-12                        # orthonormal rows
    full = np.linalg.eigvalsh(C)[::-1]
    assert _rel(w, full[:k]) < 1e-12                               # the k largest
    for r in range(k):                                             # the sign rule
        i = int(np.argmax(np.abs(P[r])))
        assert P[r, i] > 0
    # a diagonal covariance: coordinate vectors of its k largest entries, in order
    d = W.rng(19).permutation(np.arange(1.0, n + 1.0))
    Pd, wd = oracle.pca_topk(np.diag(d), k)
    top = np.argsort(-d)[:k]
    assert np.array_equal(wd, d[top])
    assert np.array_equal(Pd, np.eye(n)[top])


def test_pca_topk_kfac_kronecker_structure():
    """Sec. 3.2: eigenvectors of C_F (x) C_B are Kronecker products of the
    factors' eigenvectors, so the top eigenvectors of H_KFAC are products of
    top eigenvectors, and projecting H_KFAC with P_i (x) P_o (the PCA
    initialisation) leaves the diagonal matrix of the kept eigenvalue products."""
    nf, nb, kf, kb = 9, 6, 3, 2
    CF, CB = W.spd_matrix(20, nf, nf).astype(np.float64), W.spd_matrix(21, nb, nb).astype(np.float64)
    PF, wF = oracle.pca_topk(CF, kf)
    PB, wB = oracle.pca_topk(CB, kb)
    H = np.kron(CF, CB)
    PH, wH = oracle.pca_topk(H, 1)
    assert _rel(wH, [wF[0] * wB[0]]) < 1e-12
    assert _rel(PH[0], np.kron(PF[0], PB[0])) < 1e-10
    Pk = np.kron(PF, PB)
    assert _rel(Pk @ H @ Pk.T, np.diag(np.kron(wF, wB))) < 1e-12


def test_project_layers_form_equals_per_layer_calls():
    """The (layer, example)-parallel form computes each layer exactly as its own
    call (same per-example arithmetic; only the parallel loop differs), with
    layers of different widths and a ragged mask that empties one example."""
    lens = np.array([20, 0, 7])
    ds = [W.layer_inputs(3, j, 3, 20, ni, no, 4, 6, 1.0, 1.0, "bf16", lens)
          for j, (ni, no) in enumerate([(16, 24), (40, 8), (8, 32)])]
    gs = oracle.project_factored_layers([(d["x"], d["dy"], d["p_in"], d["p_out"]) for d in ds], ds[0]["mask"])
    for d, g in zip(ds, gs):
        assert np.array_equal(g, oracle.project_factored(d["x"], d["dy"], d["p_in"], d["p_out"], d["mask"]))
    assert np.all(gs[1][1] == 0.0)
