"""End-to-end tiny fp32 workload (one 64->64 layer, k = 8, 4 train + 2 test
examples of 16 tokens, damping 1e-3 x mean eigenvalue, scores 2 x 4, top-1):
project -> covariance -> precondition -> scores -> top-1 on the GPU, against
the same chain in float64.

Stage outputs (G, S) meet 1e-4.  The preconditioned test gradients and the
scores pass through fp32 S, and a rank-4 covariance with 1e-3 damping is
ill-conditioned (kappa ~ 1e4), so their bound is derived from the
conditioning: max(1e-4, 16 * kappa * 2^-24)."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


def tiny_inputs(seed=0):
    w = W.WORKLOADS["tiny_f32"]
    (_, n_in, n_out), = w.layers
    tr = W.layer_inputs(seed, 0, w.B, w.T, n_in, n_out, w.k_in, w.k_out, w.x_std, w.dy_std, "f32")
    te = W.layer_inputs(seed, 1, w.extra["Q"], w.T, n_in, n_out, w.k_in, w.k_out, w.x_std, w.dy_std, "f32")
    te["p_in"], te["p_out"] = tr["p_in"], tr["p_out"]   # one projection per layer
    return w, tr, te


def run_gpu(w, tr, te):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    D = w.D
    g_tr = torch.zeros((w.B, D), dtype=torch.float32, device="cuda")
    g_te = torch.zeros((w.extra["Q"], D), dtype=torch.float32, device="cuda")
    p_in, p_out = dev(tr["p_in"]), dev(tr["p_out"])
    P.logra_project_layer(dev(tr["x"]), dev(tr["dy"]), p_in, p_out, g_tr)
    P.logra_project_layer(dev(te["x"]), dev(te["dy"]), p_in, p_out, g_te)
    S = torch.zeros((D, D), dtype=torch.float32, device="cuda")
    P.logra_cov_accumulate(g_tr, S)
    pre = torch.zeros_like(g_te)
    P.logra_precondition(S, w.B, w.extra["damp"], g_te, pre)
    s = torch.zeros((w.extra["Q"], w.B), dtype=torch.float32, device="cuda")
    k = w.extra["topk"]
    tv = torch.zeros((w.extra["Q"], k), dtype=torch.float32, device="cuda")
    ti = torch.zeros((w.extra["Q"], k), dtype=torch.int64, device="cuda")
    P.logra_influence_scores(pre, g_tr, scores=s, topk=k, topk_val=tv, topk_idx=ti)
    torch.cuda.synchronize()
    return {n: host(t) for n, t in dict(g_tr=g_tr, g_te=g_te, S=S, pre=pre, s=s, tv=tv, ti=ti).items()}


def run_oracle(w, tr, te):
    g_tr = oracle.project_factored(tr["x"], tr["dy"], tr["p_in"], tr["p_out"])
    g_te = oracle.project_factored(te["x"], te["dy"], te["p_in"], te["p_out"])
    S = oracle.cov_accumulate(g_tr)
    pre, lam = oracle.precondition(S, w.B, w.extra["damp"], g_te)
    s = oracle.scores(pre, g_tr)
    tv, ti = oracle.topk(s, w.extra["topk"])
    kappa = np.linalg.cond(S / w.B + lam * np.eye(w.D))
    return dict(g_tr=g_tr, g_te=g_te, S=S, pre=pre, s=s, tv=tv, ti=ti, kappa=kappa)


def check(got, want):
    from gpu_util import normwise, rowwise_normwise
    assert rowwise_normwise(got["g_tr"], want["g_tr"]) <= 1e-4
    assert rowwise_normwise(got["g_te"], want["g_te"]) <= 1e-4
    assert normwise(got["S"], want["S"]) <= 1e-4
    tol = max(1e-4, 16 * want["kappa"] * 2.0 ** -24)
    assert rowwise_normwise(got["pre"], want["pre"]) <= tol
    ds = np.abs(got["s"] - want["s"])
    scale = np.linalg.norm(want["pre"], axis=1)[:, None] * np.linalg.norm(want["g_tr"], axis=1)[None, :]
    assert np.max(ds / scale) <= tol
    for q in range(want["s"].shape[0]):
        srt = np.sort(want["s"][q])[::-1]
        if srt[0] - srt[1] > 2 * tol * scale[q].max():
            assert got["ti"][q, 0] == want["ti"][q, 0]
    return tol


def test_tiny_end_to_end():
    from gpu_util import say
    say("[e2e] tiny fp32 workload")
    w, tr, te = tiny_inputs()
    want = run_oracle(w, tr, te)
    got = run_gpu(w, tr, te)
    tol = check(got, want)
    say(f"  kappa {want['kappa']:.3e} -> tolerance {tol:.3e}")
