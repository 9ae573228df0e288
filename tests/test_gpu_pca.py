"""GPU parity of the PCA initialisation of the projections (Sec. 3.2) against
the float64 oracle: the KFAC activation covariance (masked SYRK) and the
top-k eigenvectors.

Activation covariance: bf16 products are exact in fp32 and the sums run in
fp32, so the bar is 1e-5 normwise; integer-valued activations make every sum
exact, and the result must then equal the oracle bit for bit.  C must stay
exactly symmetric."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


def _act_cov_gpu(a, mask=None, calls=1):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    n = a.shape[2]
    C = torch.zeros((n, n), dtype=torch.float32, device="cuda")
    ad = dev(a)
    md = None if mask is None else dev(mask)
    for _ in range(calls):
        P.logra_act_cov_accumulate(ad, C, mask=md)
    torch.cuda.synchronize()
    return host(C)


COV_CASES = {
    # name: (dtype, B, T, n, masked)
    "bf16_ragged_two_tiles": ("bf16", 3, 70, 264, True),
    "bf16_unmasked_three_tiles": ("bf16", 2, 32, 640, False),
    "bf16_tiny": ("bf16", 1, 5, 8, True),
    "f32_ragged": ("f32", 2, 40, 36, True),
}


@pytest.mark.parametrize("name", sorted(COV_CASES))
def test_act_cov_parity(name):
    from gpu_util import normwise, say
    dtype, B, T, n, masked = COV_CASES[name]
    say(f"[act cov parity] case={name}")
    g = W.rng(60, B, T, n)
    a = W.normal(g, (B, T, n), 1.0, dtype)
    mask = None
    if masked:
        lens = W.lengths(g, B, 0, T)
        lens[-1] = T
        mask = W.mask_from_lengths(lens, T)
        if B > 1:
            mask[0] = 0                           # a fully masked example
        a[mask == 0] = np.uint16(0x7FC0) if dtype == "bf16" else np.nan   # never read
    got = _act_cov_gpu(a, mask)
    want = oracle.act_cov(a, mask)
    assert np.array_equal(got, got.T)
    assert np.all(np.isfinite(got))
    err = normwise(got, want)
    say(f"  normwise err {err:.2e}")
    assert err <= 1e-5


def test_act_cov_integer_exact_accumulates_and_repeats():
    from gpu_util import say
    say("[act cov] integer activations: exact, accumulated over calls, deterministic")
    g = W.rng(61)
    B, T, n = 4, 96, 520
    a = W.integer_array(g, (B, T, n), -3, 3, "bf16", 0.7)
    lens = W.lengths(g, B, 1, T)
    mask = W.mask_from_lengths(lens, T)
    want = oracle.act_cov(a, mask)
    got = _act_cov_gpu(a, mask, calls=2)
    assert np.array_equal(got.astype(np.float64), 2.0 * want)
    again = _act_cov_gpu(a, mask, calls=2)
    assert np.array_equal(got.view(np.uint32), again.view(np.uint32))


def _sym_start(g, n):
    """A symmetric fp32 starting C (the group accumulates into it)."""
    m = W.normal(g, (n, n), 1.0, "f32")
    return ((m + m.T) * 0.5).astype(np.float32)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_act_cov_group_equals_single_calls(dtype):
    """Several factors of one batch in one grouped launch (different n, one
    activation tensor feeding two factors, symmetric non-zero starting C): each
    C equals, bit for bit, what a call of its own gives, and matches the oracle."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, normwise, say
    g = W.rng(62)
    B, T = 3, 70
    ns = [264, 8, 640, 520, 264] if dtype == "bf16" else [36, 20, 36]
    say(f"[act cov group] {dtype}: B={B} T={T} n={ns}")
    lens = W.lengths(g, B, 0, T)
    lens[0], lens[-1] = 0, T                      # a fully masked example and a full one
    mask = W.mask_from_lengths(lens, T)
    acts = [W.normal(g, (B, T, n), 1.0, dtype) for n in ns[:-1]]
    acts.append(acts[0])                          # the same activations into a second C
    for a in acts[:-1]:
        a[mask == 0] = np.uint16(0x7FC0) if dtype == "bf16" else np.nan   # never read
    starts = [_sym_start(g, n) for n in ns]
    ad = [dev(a) for a in acts[:-1]]
    ad.append(ad[0])
    md = dev(mask)
    Cg = [dev(c) for c in starts]
    P.logra_act_cov_accumulate_group(list(zip(ad, Cg)), mask=md)
    Cs = [dev(c) for c in starts]
    for a, C in zip(ad, Cs):
        P.logra_act_cov_accumulate(a, C, mask=md)
    torch.cuda.synchronize()
    for i, n in enumerate(ns):
        got, single = host(Cg[i]), host(Cs[i])
        assert np.array_equal(got.view(np.uint32), single.view(np.uint32)), f"factor {i} (n={n})"
        assert np.array_equal(got, got.T)
        err = normwise(got.astype(np.float64) - starts[i], oracle.act_cov(acts[i], mask))
        say(f"  factor {i} (n={n}): equals its own call; normwise err vs oracle {err:.2e}")
        assert err <= 1e-5


def test_act_cov_group_full_table():
    """A table of LOGRA_MAX_ACT_COV_GROUP factors (n from 8 to 520, some
    1-tile, some 3-tile): every factor's workgroup slots decode to the right
    factor; each C equals its own call bit for bit."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    g = W.rng(63)
    B, T = 2, 40
    ns = [8 * (1 + (7 * i) % 65) for i in range(P.MAX_ACT_COV_GROUP)]
    say(f"[act cov group] {len(ns)} factors, n in {min(ns)}..{max(ns)}")
    mask = W.mask_from_lengths(W.lengths(g, B, 1, T), T)
    md = dev(mask)
    ad = [dev(W.normal(g, (B, T, n), 1.0, "bf16")) for n in ns]
    Cg = [torch.zeros((n, n), dtype=torch.float32, device="cuda") for n in ns]
    Cs = [torch.zeros((n, n), dtype=torch.float32, device="cuda") for n in ns]
    P.logra_act_cov_accumulate_group(list(zip(ad, Cg)), mask=md)
    for a, C in zip(ad, Cs):
        P.logra_act_cov_accumulate(a, C, mask=md)
    torch.cuda.synchronize()
    for i in range(len(ns)):
        assert torch.equal(Cg[i], Cs[i]), f"factor {i} (n={ns[i]})"
    err = np.max(np.abs(host(Cg[-1]).astype(np.float64) - oracle.act_cov(host(ad[-1]), mask)))
    assert err <= 1e-5 * max(1.0, float(np.max(np.abs(host(Cs[-1])))))


def _pca_gpu(C, k, dtype="f32", iters=30):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    n = C.shape[0]
    Pt = torch.full((k, n + 3), float("nan"), dtype=torch.float32 if dtype == "f32" else torch.bfloat16,
                    device="cuda")
    ev = torch.empty(k, dtype=torch.float32, device="cuda")
    P.logra_pca_topk(dev(C), k, Pt[:, :n], eigvals=ev, iters=iters)
    torch.cuda.synchronize()
    out = host(Pt)
    assert np.all(np.isnan(W.bf16_bits_to_f32(out[:, n:]) if dtype == "bf16" else out[:, n:]))   # nothing past n
    return out[:, :n], host(ev)


def _compare_rows(got, want, tol):
    """Rows of two eigenvector sets: equal up to the tolerance, and up to sign
    only where the sign rule's pivot is a near-tie (both sides apply it)."""
    from gpu_util import f64
    g = f64(got)
    errs = []
    for r in range(want.shape[0]):
        s = 1.0 if np.dot(g[r], want[r]) >= 0 else -1.0
        i = int(np.argmax(np.abs(want[r])))
        top2 = np.sort(np.abs(want[r]))[-2:] if want.shape[1] > 1 else np.array([0.0, 1.0])
        if s < 0:
            assert top2[1] - top2[0] <= 4 * tol, f"row {r}: sign differs without a near-tie pivot"
        errs.append(np.max(np.abs(s * g[r] - want[r])))
        assert errs[-1] <= tol, (r, errs[-1])
    return max(errs)


PCA_CASES = {
    # name: (n, k, decay, out dtype)
    "n300_k16_f32": (300, 16, 0.9, "f32"),
    "n64_k8_bf16": (64, 8, 0.8, "bf16"),
    "n20_k12_full_width": (20, 12, 0.7, "f32"),
    "n1000_k64_widest": (1000, 64, 0.95, "f32"),
    "n17_k1": (17, 1, 0.6, "f32"),
    # two column splits, n not a multiple of 4 (the last 4-column chunk of a
    # row runs past its end), subspace widths 48 and 80
    "n1101_k24_ragged_two_splits": (1101, 24, 0.9, "f32"),
    "n1500_k40_two_splits": (1500, 40, 0.95, "f32"),
    # odd subspace width p = n = 21: the Jacobi schedule pairs one index with padding
    "n21_k12_odd_width": (21, 12, 0.7, "f32"),
}


@pytest.mark.parametrize("name", sorted(PCA_CASES))
def test_pca_topk_parity(name):
    """Synthetic covariances with a geometric spectrum (gaps of 1 - decay
    between neighbours); both sides get the same fp32 C.  Eigenvector entries
    to 1e-4 (fp32 products, gaps >= 5%), 1e-2 for bf16 rows; Ritz values to
    1e-5 relative; the GPU's fp32 rows obey the sign rule exactly."""
    from gpu_util import say
    n, k, decay, dt = PCA_CASES[name]
    say(f"[pca parity] case={name}")
    C = W.spectral_matrix(62, n, decay, scale=1e3)
    got, ev = _pca_gpu(C, k, dt)
    want, wev = oracle.pca_topk(C.astype(np.float64), k)
    err = _compare_rows(got, want, 1e-4 if dt == "f32" else 1e-2)
    eerr = float(np.max(np.abs(ev - wev) / wev))
    say(f"  max entry err {err:.2e}, eigenvalue err {eerr:.2e}")
    assert eerr <= 1e-5
    if dt == "f32":
        for r in range(k):
            i = int(np.argmax(np.abs(got[r])))
            assert got[r, i] > 0


def test_pca_diagonal_covariance():
    """A diagonal covariance (entries 0.8^r in a random order, so that 30
    iterations converge): the rows are coordinate vectors of the largest
    diagonal entries, in order, with +1 at the pivot."""
    from gpu_util import say
    say("[pca] diagonal covariance")
    n, k = 50, 5
    d = W.rng(63).permutation(0.8 ** np.arange(n)).astype(np.float32)
    got, ev = _pca_gpu(np.diag(d), k)
    top = np.argsort(-d)[:k]
    assert np.allclose(got, np.eye(n, dtype=np.float32)[top], atol=1e-5)
    assert np.allclose(ev, d[top], rtol=1e-6)


def test_pca_from_masked_activations_end_to_end():
    """C_F of ragged, masked bf16 activations with a decaying spectrum on the
    GPU, then its top-16 eigenvectors, against the oracle's float64 C_F and
    eigh.  Rows are compared where the oracle's eigengaps are at least 2% of
    the eigenvalue (sin of the angle <= 1e-3)."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, f64, host, say
    say("[pca] masked activations -> C_F -> top-16")
    g = W.rng(64)
    B, T, n, k = 4, 96, 192, 16
    a = W.structured_activations(g, B, T, n, 0.9, "bf16")
    lens = W.lengths(g, B, 20, T)
    mask = W.mask_from_lengths(lens, T)
    C = torch.zeros((n, n), dtype=torch.float32, device="cuda")
    P.logra_act_cov_accumulate(dev(a), C, mask=dev(mask))
    Pt = torch.empty((k, n), dtype=torch.float32, device="cuda")
    ev = torch.empty(k, dtype=torch.float32, device="cuda")
    P.logra_pca_topk(C, k, Pt, eigvals=ev)
    torch.cuda.synchronize()
    got, ev = host(Pt), host(ev)
    Cw = oracle.act_cov(a, mask)
    want, wev = oracle.pca_topk(Cw, k)
    full = np.sort(np.linalg.eigvalsh(Cw))[::-1]
    gaps = np.minimum(full[:k] - full[1:k + 1], np.concatenate([[np.inf], full[:k - 1] - full[1:k]]))
    ok = gaps >= 0.02 * full[:k]
    say(f"  {int(ok.sum())} of {k} rows well separated")
    assert ok.sum() >= k - 1   # this seeded spectrum: 15 of 16 (one neighbour pair is under 2% apart)
    for r in np.nonzero(ok)[0]:
        s = 1.0 if np.dot(got[r], want[r]) >= 0 else -1.0
        sin = np.sqrt(max(0.0, 1.0 - float(np.dot(f64(got[r]), want[r])) ** 2))
        assert sin <= 1e-3, (r, sin)
        assert s > 0 or np.sort(np.abs(want[r]))[-1] - np.sort(np.abs(want[r]))[-2] < 1e-3
    assert np.max(np.abs(ev - wev) / wev) <= 1e-4
