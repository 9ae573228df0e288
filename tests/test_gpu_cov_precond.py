"""GPU parity of the covariance (Eq. (3), App. D) and the damped-inverse
preconditioner (Eq. (2) step (1), App. C) against the float64 oracle.

Preconditioner inputs are spectral random SPD matrices from the input
generator, so both sides consume the same fp32 bytes of S."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,B,D", [("bf16", 37, 200), ("bf16", 16, 512), ("f32", 5, 64),
                                       ("f32", 9, 100), ("bf16", 300, 64)])
def test_cov_parity_and_symmetry(dtype, B, D):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, normwise, say
    say(f"[cov parity] dtype={dtype} B={B} D={D}")
    g = W.normal(W.rng(21, B, D), (B, D), 1.0, dtype)
    S = torch.zeros((D, D), dtype=torch.float32, device="cuda")
    P.logra_cov_accumulate(dev(g), S)
    torch.cuda.synchronize()
    got = host(S)
    want = oracle.cov_accumulate(g)
    assert np.array_equal(got, got.T)          # exactly symmetric
    err = normwise(got, want)
    say(f"  normwise err {err:.3e}")
    assert err <= (1e-4 if dtype == "f32" else 2e-2)
    assert err <= 1e-5


def test_cov_integer_exact_blocks_and_chunks():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say("[cov] integer exact, blocks, chunked")
    g = W.integer_array(W.rng(22), (40, 3 * 72), -3, 3, "bf16")
    S = torch.zeros((3, 72, 72), dtype=torch.float32, device="cuda")
    gd = dev(g)
    P.logra_cov_accumulate_blocks(gd[:25], S, 72)      # chunked: 25 then 15 rows
    P.logra_cov_accumulate_blocks(gd[25:], S, 72)
    torch.cuda.synchronize()
    got = host(S)
    for l in range(3):
        want = oracle.cov_accumulate(g[:, l * 72:(l + 1) * 72])
        assert np.array_equal(got[l].astype(np.float64), want)


@pytest.mark.parametrize("B1,B2,D,nb,pad,s_shift", [
    (40, 5, 192, 2, 8, 0),     # register tiles: 3 off-diagonal + 3 diagonal per block, 2 chunks then 1
    (8, 0, 128, 1, 0, 0),      # register tiles, a single short chunk
    (33, 31, 64, 3, 16, 0),    # diagonal tiles only (one tile per block)
    (20, 12, 128, 2, 0, 1),    # S not 16-byte aligned: the general kernel
])
def test_cov_integer_exact_tile_paths(B1, B2, D, nb, pad, s_shift):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say(f"[cov] integer exact, B={B1}+{B2}, D={D}, blocks={nb}, row pad={pad}, S shift={s_shift}")
    ld = D * nb + pad
    g = W.integer_array(W.rng(24, B1, D), (B1 + B2, ld), -4, 4, "bf16")
    gd = dev(g)
    base = torch.zeros(nb * D * D + s_shift, dtype=torch.float32, device="cuda")
    S0 = W.integer_array(W.rng(25, D), (nb, D, D), -50, 50, "f32")
    S0 = S0 + S0.transpose(0, 2, 1)   # symmetric, as an accumulated S is
    base[s_shift:] = torch.from_numpy(S0.reshape(-1)).cuda()
    S = base[s_shift:].view(nb, D, D)
    for lo, hi in ((0, B1), (B1, B1 + B2)):
        if hi > lo:
            P.logra_cov_accumulate_blocks(gd[lo:hi], S, D)
    torch.cuda.synchronize()
    got = host(S)
    for l in range(nb):
        want = S0[l].astype(np.float64) + oracle.cov_accumulate(g[:, l * D:(l + 1) * D])
        assert np.array_equal(got[l].astype(np.float64), want)
        assert np.array_equal(got[l], got[l].T)


@pytest.mark.parametrize("B1,B2,D,nb,pad,dtype", [
    (40, 5, 192, 2, 8, "bf16"),    # register tiles below the diagonal + diagonal tiles, 2 chunks then 1
    (33, 0, 64, 3, 16, "bf16"),    # diagonal tiles only
    (25, 15, 72, 3, 0, "bf16"),    # ragged D: the general kernel
    (9, 4, 100, 2, 3, "f32"),      # fp32 rows: the general kernel
])
def test_cov_lower_integer_exact_upper_untouched(B1, B2, D, nb, pad, dtype):
    """Lower-triangle form (SYRK, uplo = lower): the lower triangle and diagonal
    equal the oracle's exactly; every entry above the diagonal keeps its bits."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say(f"[cov lower] integer exact, B={B1}+{B2}, D={D}, blocks={nb}, pad={pad}, {dtype}")
    ld = D * nb + pad
    g = W.integer_array(W.rng(26, B1, D), (B1 + B2, ld), -4, 4, dtype)
    gd = dev(g)
    S0 = W.integer_array(W.rng(27, D), (nb, D, D), -50, 50, "f32")
    S0 = S0 + S0.transpose(0, 2, 1)
    up = np.triu(np.ones((D, D), bool), 1)
    S0[:, up] = np.nan                      # never read: a NaN there would spread into the result
    S = dev(S0)
    for lo, hi in ((0, B1), (B1, B1 + B2)):
        if hi > lo:
            P.logra_cov_accumulate_blocks_lower(gd[lo:hi], S, D)
    torch.cuda.synchronize()
    got = host(S)
    assert np.array_equal(got[:, up].view(np.uint32), S0[:, up].view(np.uint32))
    for l in range(nb):
        want = S0[l].astype(np.float64) + oracle.cov_accumulate(g[:, l * D:(l + 1) * D])
        assert np.array_equal(got[l][~up].astype(np.float64), want[~up])


def test_precondition_and_self_influence_read_only_the_lower_triangle():
    """The statistic kept as its lower triangle feeds the preconditioner and the
    inverse factor to the same bits as the symmetric statistic."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    nb, D, B, Q = 3, 128, 300, 5
    say(f"[cov lower] preconditioner and self-influence from the lower triangle, {nb} blocks of {D}")
    g = dev(W.normal(W.rng(28), (B, nb * D), 1.0, "bf16"))
    S_full = torch.zeros((nb, D, D), dtype=torch.float32, device="cuda")
    S_low = torch.triu(torch.full((nb, D, D), float("nan"), dtype=torch.float32, device="cuda"), 1)
    P.logra_cov_accumulate_blocks(g, S_full, D)
    P.logra_cov_accumulate_blocks_lower(g, S_low, D)
    torch.cuda.synchronize()
    lo = np.tril(np.ones((D, D), bool))
    assert np.array_equal(host(S_full)[:, lo].view(np.uint32), host(S_low)[:, lo].view(np.uint32))
    gt = dev(W.normal(W.rng(29), (Q, nb * D), 1.0, "f32"))
    outs = []
    for S in (S_full, S_low):
        o = torch.empty((Q, nb * D), dtype=torch.float32, device="cuda")
        P.logra_precondition_blocks(S, B, 0.1, gt, o)
        si = torch.empty(B, dtype=torch.float32, device="cuda")
        P.logra_self_influence_blocks(S, B, 0.1, g, self_out=si)
        torch.cuda.synchronize()
        outs.append((host(o), host(si)))
    assert np.all(np.isfinite(outs[0][0])) and np.all(np.isfinite(outs[0][1]))
    assert np.array_equal(outs[0][0].view(np.uint32), outs[1][0].view(np.uint32))
    assert np.array_equal(outs[0][1].view(np.uint32), outs[1][1].view(np.uint32))


def test_cov_deterministic():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say("[cov] determinism")
    g = dev(W.normal(W.rng(23), (64, 256), 1.0, "bf16"))
    outs = []
    for _ in range(2):
        S = torch.zeros((256, 256), dtype=torch.float32, device="cuda")
        P.logra_cov_accumulate(g, S)
        torch.cuda.synchronize()
        outs.append(host(S))
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))


PRE_CASES = {
    # name: (D, rank, n_blocks, Q, damp, in_dtype, out_dtype)
    "tiny_f32": (64, 4, 1, 2, 1e-3, "f32", "f32"),
    "ragged_D": (200, 50, 1, 7, 0.1, "bf16", "f32"),
    "blocks_bf16": (256, 256, 5, 37, 0.1, "bf16", "bf16"),
    "blocks_many_q": (64, 30, 3, 70, 0.1, "f32", "f32"),
    "D1000": (1000, 1000, 1, 5, 0.1, "f32", "f32"),
}


@pytest.mark.parametrize("name", sorted(PRE_CASES))
def test_precondition_parity(name):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, rowwise_normwise, say
    D, rank, nb, Q, r, idt, odt = PRE_CASES[name]
    say(f"[precondition parity] case={name}")
    N = 4096
    S = np.stack([W.spd_matrix(30 + l, D, rank, scale=float(N)) for l in range(nb)])
    g = W.normal(W.rng(31, D), (Q, nb * D), 1.0, idt)
    out = torch.zeros((Q, nb * D), dtype=torch.float32 if odt == "f32" else torch.bfloat16, device="cuda")
    P.logra_precondition_blocks(dev(S), N, r, dev(g), out)
    got = host(out)
    want = np.concatenate([oracle.precondition(S[l].astype(np.float64), N, r, g[:, l * D:(l + 1) * D])[0]
                           for l in range(nb)], axis=1)
    tol = 1e-4 if odt == "f32" else 2e-2
    for l in range(nb):
        err = rowwise_normwise(got[:, l * D:(l + 1) * D], want[:, l * D:(l + 1) * D])
        say(f"  block {l}: normwise err {err:.3e} (tol {tol})")
        assert err <= tol


def test_precondition_identity_and_single_api():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say("[precondition] identity mode, single-block API")
    g = W.normal(W.rng(32), (3, 64), 1.0, "bf16")
    out = torch.zeros((3, 64), dtype=torch.float32, device="cuda")
    S = torch.zeros((64, 64), dtype=torch.float32, device="cuda")
    P.logra_precondition(S, 1, -1.0, dev(g), out)
    assert np.array_equal(host(out), W.bf16_bits_to_f32(g))


def test_precondition_not_pd():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, say
    say("[precondition] not positive definite")
    v = np.zeros((1, 64), np.float32)
    v[0, :2] = [1.0, 2.0]
    S = np.outer(v[0], v[0]).astype(np.float32)   # rank one: second pivot is exactly zero
    out = torch.zeros((1, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(P.LograError) as ei:
        P.logra_precondition(dev(S), 1, 0.0, dev(v), out)
    assert ei.value.status == P.ERR_NOT_PD
    S2 = np.eye(64, dtype=np.float32)
    S2[10, 10] = -1.0
    with pytest.raises(P.LograError) as ei:
        P.logra_precondition(dev(S2), 1, 0.0, dev(v), out)
    assert ei.value.status == P.ERR_NOT_PD
    assert "pivot 10" in P.logra_last_error()
