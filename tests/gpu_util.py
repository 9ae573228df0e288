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
