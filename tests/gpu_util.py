"""Host/device marshalling and error metrics for the GPU parity tests."""
import numpy as np

import workloads as W

DEV = "cuda:0"


def dev(a):
    """numpy -> device tensor (uint16 arrays are bf16 bit patterns)."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(a.copy()).to(DEV)


def host(t):
    """device tensor -> numpy (bf16 as uint16 bit patterns)."""
    import torch
    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def f64(a):
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return W.bf16_bits_to_f32(a).astype(np.float64)
    return a.astype(np.float64)


def normwise(got, want):
    """max |got - want| / max |want| (0 when both are zero)."""
    got, want = f64(got), f64(want)
    den = np.abs(want).max() if want.size else 0.0
    num = np.abs(got - want).max() if want.size else 0.0
    if den == 0.0:
        return 0.0 if num == 0.0 else np.inf
    return float(num / den)


def rowwise_normwise(got, want):
    """Worst normwise error over rows (one row = one example / query)."""
    got, want = f64(got), f64(want)
    return max((normwise(got[i], want[i]) for i in range(want.shape[0])), default=0.0)


def empty(shape, dtype):
    import torch
    return torch.empty(shape, dtype=dtype, device=DEV)


def zeros(shape, dtype):
    import torch
    return torch.zeros(shape, dtype=dtype, device=DEV)


def say(*a):
    print(*a, flush=True)


def topk_agreement(got_idx, want_row, tau, k):
    """Top-k parity where several answers are correct (near-ties).

    got_idx: the GPU's top-k indices of one query (sorted by its scores);
    want_row: the oracle's float64 scores of the whole row; tau: per-index
    tolerance of a score (array over the row).  Checks that
      - the rank-r index is the oracle's wherever the oracle's rank-r score
        is separated from both neighbours by more than their tolerances;
      - an index in one top-k set but not the other lies within tolerance
        of the oracle's k-th score (a near-tie at the boundary).
    Returns (ranks checked, boundary swaps)."""
    n = want_row.shape[0]
    order = np.lexsort((np.arange(n), -want_row))[:k + 1]
    s = want_row[order]
    checked = 0
    for r in range(min(k, n)):
        above = r == 0 or s[r - 1] - s[r] > tau[order[r - 1]] + tau[order[r]]
        below = r + 1 >= len(order) or s[r] - s[r + 1] > tau[order[r]] + tau[order[r + 1]]
        if above and below:
            assert got_idx[r] == order[r], f"rank {r}: {got_idx[r]} != oracle {order[r]}"
            checked += 1
    kth = order[min(k, n) - 1]
    swaps = set(int(j) for j in got_idx) ^ set(int(j) for j in order[:k])
    for j in swaps:
        assert abs(want_row[j] - want_row[kth]) <= tau[j] + tau[kth], f"index {j} is not a boundary near-tie"
    return checked, len(swaps) // 2
