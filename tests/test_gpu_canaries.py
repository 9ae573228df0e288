"""Guard bands around every output buffer of every entry point: each output is
an interior window of a larger device buffer filled with a sentinel bit
pattern, at an odd row stride where the call allows one; after the call the
bytes before, after and between the rows must still hold the sentinel, so an
out-of-range store anywhere shows up here (the stores themselves are checked
against the oracle by the parity tests)."""
import ctypes

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

GUARD = 4096          # guard band in elements on each side
SENT32 = 0x7FA5A5A5   # a NaN pattern no result takes
SENT16 = 0x7FA5


def _guarded(torch, rows, cols, ld, dtype):
    """(full buffer, interior view [rows, cols] at row stride ld) with sentinels everywhere."""
    itemsize = torch.tensor([], dtype=dtype).element_size()
    n = 2 * GUARD + rows * ld
    if itemsize == 2:
        full = torch.full((n,), SENT16 - 65536 if SENT16 > 32767 else SENT16, dtype=torch.int16, device="cuda")
    elif itemsize == 4:
        full = torch.full((n,), SENT32, dtype=torch.int32, device="cuda")
    else:
        full = torch.full((n,), (SENT32 << 32) | SENT32, dtype=torch.int64, device="cuda")
    view = full.view(dtype)[GUARD:GUARD + rows * ld].view(rows, ld)[:, :cols]
    return full, view


def _check(full, rows, cols, ld, what):
    from gpu_util import host
    h = host(full).view(np.uint16 if full.element_size() == 2 else np.uint32 if full.element_size() == 4 else np.uint64)
    sent = {2: SENT16, 4: SENT32, 8: (SENT32 << 32) | SENT32}[full.element_size()]
    assert np.all(h[:GUARD] == sent), f"{what}: store before the buffer"
    assert np.all(h[GUARD + rows * ld:] == sent), f"{what}: store after the buffer"
    body = h[GUARD:GUARD + rows * ld].reshape(rows, ld)
    assert np.all(body[:, cols:] == sent), f"{what}: store between rows"
    assert not np.any(body[:, :cols] == sent), f"{what}: an output element was not written"


def test_canaries_projection_and_covariance():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, say
    say("[canary] projection (k = 16 per-wave path, k = 64 tile groups, no-alloc), covariance fp32 / fp64")
    for k, dt in ((16, torch.bfloat16), (64, torch.float32), (24, torch.bfloat16)):
        B, T, n_in, n_out = 5, 150, 520, 776
        d = W.layer_inputs(3, k, B, T, n_in, n_out, k, k, 1.0, 1.0, "bf16", np.array([150, 0, 3, 64, 77]))
        D = k * k
        ld = D + 13
        full, g = _guarded(torch, B, D, ld, dt)
        P.logra_project_layer(dev(d["x"]), dev(d["dy"]), dev(d["p_in"]), dev(d["p_out"]), g, mask=dev(d["mask"]))
        torch.cuda.synchronize()
        _check(full, B, D, ld, f"projection k={k}")
    d = W.layer_inputs(4, 1, 3, 90, 256, 128, 16, 16, 1.0, 1.0, "bf16")
    full, g = _guarded(torch, 3, 256, 256 + 8, torch.bfloat16)
    P.logra_project_layers_noalloc([dict(x=dev(d["x"]), dy=dev(d["dy"]), p_in=dev(d["p_in"]), p_out=dev(d["p_out"]),
                                         g_out=g)])
    torch.cuda.synchronize()
    _check(full, 3, 256, 264, "no-alloc projection")
    for dtype, fn in ((torch.float32, P.logra_cov_accumulate), (torch.float64, P.logra_cov_accumulate_f64)):
        D = 200
        rows = W.normal(W.rng(5), (9, D), 1.0, "f32" if dtype == torch.float64 else "bf16")
        full, S = _guarded(torch, D, D, D, dtype)
        S.zero_()
        fn(dev(rows), S)
        torch.cuda.synchronize()
        h = full.view(dtype)[GUARD:GUARD + D * D]
        assert not torch.isnan(h).any()
        side = torch.cat([full[:GUARD], full[GUARD + D * D:]]).cpu().numpy()
        assert np.all(side.view(np.uint32 if dtype == torch.float32 else np.uint64) ==
                      (SENT32 if dtype == torch.float32 else (SENT32 << 32) | SENT32)), f"covariance {dtype}"


def test_canaries_precondition_scores_topk_selfinf():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, say
    say("[canary] preconditioner, scores (bf16 filtered, fp64 accumulation), top-k, self-influence")
    D, nb, Q, N, k = 64, 3, 70, 9000, 17
    S = np.stack([W.spd_matrix(40 + l, D, D, scale=100.0) for l in range(nb)])
    te = W.normal(W.rng(6), (Q, nb * D), 1.0, "bf16")
    tr = W.normal(W.rng(7), (N, nb * D), 1.0, "bf16")
    ld = nb * D + 24
    full, pre = _guarded(torch, Q, nb * D, ld, torch.bfloat16)
    P.logra_precondition_blocks(dev(S), 100, 0.1, dev(te), pre)
    _check(full, Q, nb * D, ld, "precondition")
    ls = N + 5
    fs, s = _guarded(torch, Q, N, ls, torch.float32)
    fv, tv = _guarded(torch, Q, k, k, torch.float32)
    fi, ti = _guarded(torch, Q, k, k, torch.int64)
    P.logra_influence_scores(pre, dev(tr), scores=s, topk=k, topk_val=tv.contiguous().view(Q, k),
                             topk_idx=ti.contiguous().view(Q, k))
    torch.cuda.synchronize()
    _check(fs, Q, N, ls, "scores (filtered top-k launch)")
    _check(fv, Q, k, k, "top-k values")
    _check(fi, Q, k, k, "top-k indices")
    f64s, s64 = _guarded(torch, 3, 500, 509, torch.float32)
    te64 = torch.from_numpy(W.normal(W.rng(8), (3, 40), 1.0, "f32").astype(np.float64)).cuda()
    tr32 = torch.from_numpy(W.normal(W.rng(9), (500, 40), 1.0, "f32")).cuda()
    P.logra_influence_scores(te64, tr32, scores=s64)
    torch.cuda.synchronize()
    _check(f64s, 3, 500, 509, "fp64-accumulated scores")
    fself, self_out = _guarded(torch, 1, 4000, 4000, torch.float32)
    P.logra_self_influence_blocks(dev(S), 100, 0.1, dev(tr[:4000]), self_out=self_out.view(4000))
    torch.cuda.synchronize()
    _check(fself, 1, 4000, 4000, "self-influence")


def test_canaries_pca():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, say
    say("[canary] activation covariance and PCA rows")
    a = W.structured_activations(W.rng(10), 2, 70, 136, 0.9, "bf16")
    fc, C = _guarded(torch, 136, 136, 136, torch.float32)
    C.zero_()
    P.logra_act_cov_accumulate(dev(a), C)
    torch.cuda.synchronize()
    side = torch.cat([fc[:GUARD], fc[GUARD + 136 * 136:]]).cpu().numpy().view(np.uint32)
    assert np.all(side == SENT32), "activation covariance"
    fp, Pt = _guarded(torch, 8, 136, 136 + 8, torch.bfloat16)
    P.logra_pca_topk(C, 8, Pt, iters=10)
    torch.cuda.synchronize()
    _check(fp, 8, 136, 144, "pca rows")
