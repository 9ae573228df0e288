"""GPU parity of the float64 statistics path of fp32 workloads against the
oracle: the covariance kept in float64 (Eq. (3), App. D), the damped inverse
from an fp64 S with fp64 output (Eq. (2) step (1), App. C), and scores
accumulated in float64 (Eq. (2) step (2)) from any mix of fp32 and fp64
operands.

Both sides take the same fp32 / fp64 bytes.  Products of fp32 values are
exact in float64, so the covariance differs from the oracle's only by the
order of its float64 sums (bound: about B * 2^-53 of the largest entry); the
solve by about cond(C + lambda I) * 2^-53; a score, rounded once to fp32,
by half an fp32 ulp plus the float64 sum's rounding."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,B,D,nb", [("f32", 37, 200, 2), ("f32", 4, 64, 1), ("f64", 9, 100, 3),
                                          ("f32", 300, 72, 1)])
def test_cov_f64_parity(dtype, B, D, nb):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, normwise, say
    say(f"[cov f64] rows {dtype} B={B} D={D} blocks={nb}")
    g = W.normal(W.rng(51, B, D, nb), (B, nb * D), 1.0, "f32")
    if dtype == "f64":
        g = g.astype(np.float64) * (1.0 + 1e-9 * W.normal(W.rng(52), g.shape, 1.0, "f32").astype(np.float64))
    S = torch.zeros((nb, D, D), dtype=torch.float64, device="cuda")
    gd = dev(g)
    P.logra_cov_accumulate_f64(gd[: B // 2], S)          # chunked: two calls
    P.logra_cov_accumulate_f64(gd[B // 2:], S)
    torch.cuda.synchronize()
    got = host(S)
    for l in range(nb):
        want = oracle.cov_accumulate(np.ascontiguousarray(g[:, l * D:(l + 1) * D]))
        assert np.array_equal(got[l], got[l].T)           # exactly symmetric
        err = normwise(got[l], want)
        say(f"  block {l}: normwise err {err:.3e}")
        assert err <= 1e-13


def test_cov_f64_integer_exact():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say("[cov f64] integer rows: exact")
    g = W.integer_array(W.rng(53), (50, 2 * 64), -50, 50, "f32")
    S = torch.zeros((2, 64, 64), dtype=torch.float64, device="cuda")
    P.logra_cov_accumulate_f64(dev(g), S)
    torch.cuda.synchronize()
    got = host(S)
    for l in range(2):
        assert np.array_equal(got[l], oracle.cov_accumulate(np.ascontiguousarray(g[:, l * 64:(l + 1) * 64])))


@pytest.mark.parametrize("in_dt,out_dt", [("f32", "f64"), ("f64", "f64"), ("f32", "f32"), ("bf16", "bf16")])
def test_precondition_f64_parity(in_dt, out_dt):
    """fp64 S of a rank-deficient covariance, lightly damped (condition number
    up to ~1e5): the fp64 output matches the oracle to ~cond * 2^-53."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, rowwise_normwise, say
    D, nb, Q, N, r = 96, 2, 13, 40, 1e-3
    say(f"[precondition f64] in={in_dt} out={out_dt} D={D} blocks={nb} Q={Q}")
    gs = W.normal(W.rng(54), (N, nb * D), 1.0, "f32").astype(np.float64)
    S = np.stack([gs[:, l * D:(l + 1) * D].T @ gs[:, l * D:(l + 1) * D] for l in range(nb)])
    g = W.normal(W.rng(55), (Q, nb * D), 1.0, "f32" if in_dt != "bf16" else "bf16")
    if in_dt == "f64":
        g = g.astype(np.float64) / 3.0
    tdt = {"f32": torch.float32, "f64": torch.float64, "bf16": torch.bfloat16}[out_dt]
    out = torch.zeros((Q, nb * D), dtype=tdt, device="cuda")
    P.logra_precondition_f64(dev(S), N, r, dev(g), out)
    got = host(out)
    tol = {"f64": 1e-10, "f32": 1e-6, "bf16": 2e-2}[out_dt]
    for l in range(nb):
        want, lam = oracle.precondition(S[l], N, r, np.ascontiguousarray(g[:, l * D:(l + 1) * D]))
        kappa = np.linalg.cond(S[l] / N + lam * np.eye(D))
        err = rowwise_normwise(got[:, l * D:(l + 1) * D], want)
        say(f"  block {l}: kappa {kappa:.2e}, normwise err {err:.3e} (tol {tol})")
        assert err <= tol


@pytest.mark.parametrize("te_dt,tr_dt,Q,N,D", [("f64", "f32", 2, 4, 64), ("f32", "f32", 70, 130, 100),
                                               ("f64", "f64", 65, 257, 36), ("f32", "f64", 3, 1000, 520)])
def test_scores_f64_accumulation(te_dt, tr_dt, Q, N, D):
    """Scores of strongly cancelling operands: each is within half an fp32 ulp
    of the exact float64 score (plus the float64 sum's own rounding), and the
    top-k equals the oracle's wherever the gaps exceed that."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say(f"[scores f64 acc] te={te_dt} tr={tr_dt} Q={Q} N={N} D={D}")
    g = W.rng(56, Q, N, D)
    te = W.normal(g, (Q, D), 1.0, "f32").astype(np.float64 if te_dt == "f64" else np.float32)
    tr = W.normal(g, (N, D), 1.0, "f32").astype(np.float64 if tr_dt == "f64" else np.float32)
    if te_dt == "f64":
        te = te * 1e3 + 1e-4 * W.normal(g, (Q, D), 1.0, "f32").astype(np.float64)   # below fp32 resolution
    k = min(5, N)
    s = torch.full((Q, N), np.nan, dtype=torch.float32, device="cuda")
    tv = torch.empty((Q, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((Q, k), dtype=torch.int64, device="cuda")
    P.logra_influence_scores(dev(te), dev(tr), scores=s, topk=k, topk_val=tv, topk_idx=ti)
    torch.cuda.synchronize()
    got = host(s).astype(np.float64)
    want = oracle.scores(te, tr)
    absterm = np.abs(te.astype(np.float64)) @ np.abs(tr.astype(np.float64)).T
    bound = 2.0 ** -24 * np.abs(want) + 4 * D * 2.0 ** -53 * absterm
    excess = np.abs(got - want) / bound
    say(f"  max |ds| / bound {excess.max():.3f}")
    assert (excess <= 1.0).all()
    wv, wi = oracle.topk(want, k)
    gi = host(ti)
    for q in range(Q):
        for r in range(k):
            nxt = wv[q, r + 1] if r + 1 < k else np.sort(want[q])[::-1][k] if N > k else -np.inf
            if wv[q, r] - nxt > 2 * bound[q].max():
                assert gi[q, r] == wi[q, r]
