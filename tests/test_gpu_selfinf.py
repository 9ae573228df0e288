"""GPU parity of the l-RelatIF normalisation (Sec. 4.2): the self-influence
g^T (C + lambda I)^{-1} g of every gradient summed over the Hessian's blocks,
and influence scores scaled per query and per training example (l-RelatIF
divides by sqrt(self_train); the cosine form also by sqrt(self_test)), with
the top-k taken over the scaled scores.

Tolerances: self-influence 1e-4 relative per gradient (the inverse Cholesky
factor is applied as two bf16 halves carrying about 16 significant bits,
2^-17 per element, with fp32 accumulation; the damped spectra here keep
|W||g| within a small multiple of |Wg|; errors of about 1e-6 are typical);
1e-5 in identity mode, where the factor is exactly I and only the fp32
summation rounds.  Scaled scores: the unscaled score tolerance, 1e-3 of
|g_te||g_tr|, times the two scales.  With integer gradients and power-of-two
scales every scaled score is exact in fp32, so the top-k (with exact ties,
through the candidate-filter path) must equal the oracle's bit for bit."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

N_COV = 4096


def _spd_blocks(seed, D, nb, rank=None):
    return np.stack([W.spd_matrix(seed + l, D, rank or D, scale=float(N_COV)) for l in range(nb)])


def _self_gpu(S, damp, g, ld=None):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    rows = g.shape[0]
    gd = dev(g)
    if ld is not None:
        gd = gd[:, :ld]
    so = torch.full((rows + 1,), np.nan, dtype=torch.float32, device="cuda")
    ro = torch.full((rows + 1,), np.nan, dtype=torch.float32, device="cuda")
    P.logra_self_influence_blocks(dev(S), N_COV, damp, gd, self_out=so[:rows], rsqrt_out=ro[:rows])
    torch.cuda.synchronize()
    so, ro = host(so), host(ro)
    assert np.isnan(so[rows]) and np.isnan(ro[rows])     # nothing written past `rows`
    return so[:rows], ro[:rows]


SELF_CASES = {
    # name: (dtype, D, n_blocks, rows, extra_ld, damp)
    "bf16_D256_ragged_rows": ("bf16", 256, 3, 600, 0, 0.1),
    "bf16_D96_zero_pad_rows": ("bf16", 96, 2, 300, 0, 0.1),
    "bf16_D320_two_passes": ("bf16", 320, 1, 257, 0, 1e-2),
    "bf16_D32_one_row": ("bf16", 32, 5, 1, 0, 0.1),
    "bf16_strided_rows": ("bf16", 64, 2, 130, 72, 0.1),
    "bf16_D40_rowwise": ("bf16", 40, 2, 50, 0, 0.1),
    "f32_D48_rowwise": ("f32", 48, 3, 33, 0, 0.1),
}


@pytest.mark.parametrize("name", sorted(SELF_CASES))
def test_self_influence_parity(name):
    from gpu_util import f64, say
    dtype, D, nb, rows, extra, damp = SELF_CASES[name]
    say(f"[self-influence parity] case={name}")
    S = _spd_blocks(50, D, nb)
    ld = nb * D + extra
    gfull = W.normal(W.rng(51, D, nb, rows), (rows, ld), 1.0, dtype)
    g = np.ascontiguousarray(gfull[:, :nb * D])
    got, rs = _self_gpu(S, damp, gfull, ld=nb * D if extra else None)
    want = oracle.self_influence_blocks(S.astype(np.float64), N_COV, damp, g)
    err = np.max(np.abs(f64(got) - want) / want)
    say(f"  max relative err {err:.3e}")
    assert err <= 1e-4
    # the reciprocal square root is taken from the fp32 self-influence
    assert np.allclose(rs, 1.0 / np.sqrt(got.astype(np.float64)), rtol=1e-6, atol=0)


def test_self_influence_identity_and_zero_rows():
    """Identity mode (negative damping ratio): self = |g|^2 up to fp32
    summation; a zero gradient has self 0 and a reciprocal of 0."""
    from gpu_util import f64, say
    say("[self-influence] identity mode, zero rows")
    for D, nb, dtype in ((64, 3, "bf16"), (40, 2, "f32")):
        g = W.normal(W.rng(52, D), (70, nb * D), 1.0, dtype)
        g[5] = 0
        got, rs = _self_gpu(np.zeros((nb, D, D), np.float32), -1.0, g)
        want = np.sum(f64(g) ** 2, axis=1)
        err = np.max(np.abs(f64(got) - want) / np.maximum(want, 1e-30))
        say(f"  D={D} nb={nb} {dtype}: max relative err {err:.3e}")
        assert err <= 1e-5
        assert got[5] == 0.0 and rs[5] == 0.0


def test_self_influence_not_pd_and_empty():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, say
    say("[self-influence] not positive definite, no rows")
    S = np.stack([np.eye(64, dtype=np.float32)] * 2)
    S[1, 7, 7] = -1.0
    g = dev(W.normal(W.rng(53), (4, 128), 1.0, "bf16"))
    out = torch.zeros(4, dtype=torch.float32, device="cuda")
    with pytest.raises(P.LograError) as ei:
        P.logra_self_influence_blocks(dev(S), 1, 0.0, g, self_out=out)
    assert ei.value.status == P.ERR_NOT_PD
    assert "block 1" in P.logra_last_error() and "pivot 7" in P.logra_last_error()
    S[1, 7, 7] = 1.0
    P.logra_self_influence_blocks(dev(S), 1, 0.0, g[:0], self_out=out[:0])   # no rows: a no-op
    P.logra_self_influence_blocks(dev(S), 1, 0.0, g, self_out=out)           # the status words were reset
    torch.cuda.synchronize()
    from gpu_util import f64, host
    assert np.allclose(host(out), np.sum(f64(host(g)) ** 2, axis=1), rtol=1e-5)   # S = I, N = 1, no damping


def _scaled_gpu(te, tr, row_scale, col_scale, topk=0, materialize=True, chunks=None):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    Q, N = te.shape[0], tr.shape[0]
    ted, trd = dev(te), dev(tr)
    rsd = None if row_scale is None else dev(row_scale.astype(np.float32))
    csd = None if col_scale is None else dev(col_scale.astype(np.float32))
    s = torch.full((Q, N), np.nan, dtype=torch.float32, device="cuda") if materialize else None
    tv = torch.empty((Q, max(topk, 1)), dtype=torch.float32, device="cuda")
    ti = torch.empty((Q, max(topk, 1)), dtype=torch.int64, device="cuda")
    for c, (a, b) in enumerate(chunks or [(0, N)]):
        P.logra_influence_scores(ted, trd[a:b], scores=None if s is None else s[:, a:b], topk=topk,
                                 topk_val=tv if topk else None, topk_idx=ti if topk else None, train_base=a,
                                 merge=c > 0, row_scale=rsd,
                                 col_scale=None if csd is None else csd[a:b])
    torch.cuda.synchronize()
    return (None if s is None else host(s)), host(tv), host(ti)


@pytest.mark.parametrize("dtype,Q,N,D,mode", [("bf16", 37, 1000, 576, "relatif"), ("bf16", 37, 1000, 576, "cosine"),
                                              ("bf16", 20, 300, 192, "row_only"), ("f32", 9, 130, 36, "cosine")])
def test_scaled_scores_parity(dtype, Q, N, D, mode):
    """Scales from oracle self-influences (host-computed) against the oracle's
    normalised scores."""
    from gpu_util import f64, say
    say(f"[scaled scores] dtype={dtype} Q={Q} N={N} D={D} mode={mode}")
    g = W.rng(54, Q, N, D)
    te = W.normal(g, (Q, D), 1.0, dtype)
    tr = W.normal(g, (N, D), 1.0, dtype)
    S = _spd_blocks(55, D, 1)[0].astype(np.float64)
    self_te = oracle.self_influence(S, N_COV, 0.1, te)
    self_tr = oracle.self_influence(S, N_COV, 0.1, tr)
    rs = (1.0 / np.sqrt(self_te)) if mode in ("cosine", "row_only") else None
    cs = (1.0 / np.sqrt(self_tr)) if mode in ("cosine", "relatif") else None
    got, _, _ = _scaled_gpu(te, tr, rs, cs)
    want = oracle.scores(te, tr)
    if mode == "row_only":
        want = want / np.sqrt(self_te)[:, None]
    else:
        want = oracle.normalise_scores(want, self_tr, self_te if mode == "cosine" else None)
    bound = np.outer(np.linalg.norm(f64(te), axis=1), np.linalg.norm(f64(tr), axis=1))
    bound *= (1.0 if rs is None else rs[:, None]) * (1.0 if cs is None else cs[None, :])
    err = float(np.max(np.abs(f64(got) - want) / bound))
    say(f"  normalised err {err:.3e}")
    assert err <= 1e-3


def test_scaled_topk_integer_exact_filtered():
    """Integer gradients and power-of-two scales: every scaled score is exact,
    with many ties.  The top-k -- through the candidate filter, whose second
    launch starts past the chunk's prefix and must index the column scales
    from there -- equals the oracle's, alone and merged over chunks."""
    from gpu_util import f64, say
    say("[scaled top-k] integer scores, power-of-two scales, filtered path")
    g = W.rng(56)
    Q, N, D, k = 9, 24_000, 64, 37
    te = W.integer_array(g, (Q, D), -2, 2, "bf16", 0.5)
    tr = W.integer_array(g, (N, D), -2, 2, "bf16", 0.5)
    cs = np.exp2(g.integers(-2, 3, size=N)).astype(np.float64)     # 1/4 .. 4
    rs = np.exp2(g.integers(-1, 2, size=Q)).astype(np.float64)
    want = oracle.normalise_scores(oracle.scores(te, tr), 1.0 / cs ** 2, 1.0 / rs ** 2)
    wv, wi = oracle.topk(want, k)
    s, _, _ = _scaled_gpu(te, tr, rs, cs)                           # unfiltered: one launch over the chunk
    assert np.array_equal(f64(s), want)
    _, tv, ti = _scaled_gpu(te, tr, rs, cs, topk=k, materialize=False)
    assert np.array_equal(ti, wi)
    assert np.array_equal(tv.astype(np.float64), wv)
    _, tv2, ti2 = _scaled_gpu(te, tr, rs, cs, topk=k, materialize=False, chunks=[(0, 9_000), (9_000, 24_000)])
    assert np.array_equal(ti2, wi)
    assert np.array_equal(tv2, tv)


def test_relatif_end_to_end():
    """The whole l-RelatIF query on the GPU -- precondition the test gradients,
    self-influence of the training gradients, scaled scores with top-k --
    against the oracle's normalised scores; the top-k is the exact top-k of the
    GPU's own normalised score rows, and agrees with the oracle's wherever the
    score gaps exceed the tolerance."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, f64, host, say
    say("[l-RelatIF end to end] 2 blocks of 64, Q=16, N=9000, top-20")
    D, nb, Q, N, k, damp = 64, 2, 16, 9000, 20, 0.1
    S = _spd_blocks(57, D, nb)
    g = W.rng(58)
    te = W.normal(g, (Q, nb * D), 1.0, "bf16")
    tr = W.normal(g, (N, nb * D), 1.0, "bf16")
    Sd = dev(S)
    pre = torch.empty((Q, nb * D), dtype=torch.bfloat16, device="cuda")
    P.logra_precondition_blocks(Sd, N_COV, damp, dev(te), pre)
    rsq = torch.empty(N, dtype=torch.float32, device="cuda")
    P.logra_self_influence_blocks(Sd, N_COV, damp, dev(tr), rsqrt_out=rsq)
    s = torch.empty((Q, N), dtype=torch.float32, device="cuda")
    tv = torch.empty((Q, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((Q, k), dtype=torch.int64, device="cuda")
    P.logra_influence_scores(pre, dev(tr), scores=s, topk=0, col_scale=rsq)
    P.logra_influence_scores(pre, dev(tr), topk=k, topk_val=tv, topk_idx=ti, col_scale=rsq)
    torch.cuda.synchronize()
    s, tv, ti, pre_h = host(s), host(tv), host(ti), host(pre)
    S64 = S.astype(np.float64)
    te_pre = np.concatenate([oracle.precondition(S64[l], N_COV, damp, te[:, l * D:(l + 1) * D])[0]
                             for l in range(nb)], axis=1)
    self_tr = oracle.self_influence_blocks(S64, N_COV, damp, tr)
    want = oracle.normalise_scores(oracle.scores(te_pre, tr), self_tr)
    # the bf16 rounding of the preconditioned test gradients (at most 2^-9 per
    # element, so at most 2^-9 of |g_te,pre| |g_tr| on a score) dominates; held to
    # the stated 1e-3 of |g_te,pre| |g_tr| / sqrt(self_tr) (measured 6.9e-4)
    base = np.outer(np.linalg.norm(te_pre, axis=1), np.linalg.norm(f64(tr), axis=1) / np.sqrt(self_tr))
    err = float(np.max(np.abs(f64(s) - want) / base))
    say(f"  normalised err {err:.3e}")
    assert err <= 1e-3
    tau = 1e-3 * base
    wv, wi = oracle.topk(want, k + 1)
    checked = 0
    for q in range(Q):
        order = np.lexsort((np.arange(N), -s[q].astype(np.float64)))[:k]
        assert np.array_equal(ti[q], order) and np.array_equal(tv[q], s[q, order])
        for r in range(k):
            t = tau[q, wi[q, r]]
            lo_gap = wv[q, r] - wv[q, r + 1]
            hi_gap = wv[q, r - 1] - wv[q, r] if r > 0 else np.inf
            if lo_gap > t + tau[q, wi[q, r + 1]] and hi_gap > t + (tau[q, wi[q, r - 1]] if r > 0 else 0):
                assert ti[q, r] == wi[q, r], (q, r)
                checked += 1
    say(f"  {checked} of {Q * k} ranks resolvable, all agree")
    assert checked > 0
