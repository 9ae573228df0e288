"""The projection entry point that allocates nothing (logra_project_layers_noalloc,
for callers that cannot allocate) against the one with a caller workspace
(logra_project_layers), through the C ABI: the same kernels on the same inputs,
so the stores must agree bit for bit.  Two calls in a row on the same GPU,
the second with a smaller batch (the static workspace keeps the first call's
contents), then a batch too large for the static workspace."""
import ctypes

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


def _case(seed, layers, B, T, k, lens=None):
    import torch
    from gpu_util import dev
    out = []
    for j, (n_in, n_out) in enumerate(layers):
        d = W.layer_inputs(seed, j, B, T, n_in, n_out, k, k, 1.0, 1e-3, "bf16", lens)
        out.append(dict(x=dev(d["x"]), dy=dev(d["dy"]), p_in=dev(d["p_in"]), p_out=dev(d["p_out"])))
    mask = None if lens is None else torch.from_numpy(W.mask_from_lengths(lens, T)).cuda()
    return out, mask


def _descs(P, layers, store, D):
    arr = (P.LayerDesc * len(layers))()
    for j, L in enumerate(layers):
        g = store[:, j * D:(j + 1) * D]
        arr[j] = P.LayerDesc(L["x"].data_ptr(), L["dy"].data_ptr(), L["p_in"].data_ptr(), L["p_out"].data_ptr(),
                             g.data_ptr(), L["x"].shape[2], L["dy"].shape[2])
    return arr


def _both(layers, mask, B, T, k, g_dtype):
    """(store from logra_project_layers, store from logra_project_layers_noalloc)."""
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import host
    lib = P.lib()
    D = k * k
    tdt = torch.bfloat16 if g_dtype == P.BF16 else torch.float32
    n = len(layers)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    mp = ctypes.c_void_p(mask.data_ptr()) if mask is not None else None
    ref = torch.full((B, n * D + 8), 3.0, dtype=tdt, device="cuda")
    got = torch.full((B, n * D + 8), 3.0, dtype=tdt, device="cuda")
    da = _descs(P, layers, ref, D)
    wsb = lib.logra_project_layers_ws_size(da, n, B, T, k, k)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    rc = lib.logra_project_layers(da, n, P.BF16, B, T, mp, k, k, g_dtype, ref.stride(0), ctypes.c_void_p(ws.data_ptr()),
                                  wsb, stream)
    assert rc == P.OK, P.logra_last_error()
    db = _descs(P, layers, got, D)
    rc = lib.logra_project_layers_noalloc(db, n, P.BF16, B, T, mp, k, k, g_dtype, got.stride(0), stream)
    assert rc == P.OK, P.logra_last_error()
    torch.cuda.synchronize()
    return host(ref), host(got), wsb


def test_noalloc_matches_workspace_entry_point_twice():
    import paper_2405_13954_amd as P
    from gpu_util import say
    # call 1: three layers, ragged batch of 8 x 512, k = 16, bf16 store
    B, T, k = 8, 512, 16
    lens = W.lengths(W.rng(71), B, 1, T)
    layers, mask = _case(71, [(768, 2304), (768, 768), (3072, 768)], B, T, k, lens)
    say(f"[noalloc] call 1: 3 layers, B={B} T={T} k={k}, ragged, bf16 store")
    ref, got, wsb = _both(layers, mask, B, T, k, P.BF16)
    say(f"  workspace {wsb / 2**20:.1f} MiB of {P.NOALLOC_WS_BYTES / 2**20:.0f}")
    assert wsb <= P.NOALLOC_WS_BYTES
    assert np.array_equal(ref, got)
    assert (got[:, -8:] == ref[:, -8:]).all()        # columns past the layers untouched
    # call 2: smaller batch, other widths, k = 8, no mask, fp32 store: the static
    # workspace still holds call 1's partials and tile list
    B2, T2, k2 = 3, 100, 8
    layers2, _ = _case(72, [(256, 512), (512, 128)], B2, T2, k2)
    say(f"[noalloc] call 2: 2 layers, B={B2} T={T2} k={k2}, unmasked, fp32 store")
    ref2, got2, _ = _both(layers2, None, B2, T2, k2, P.F32)
    assert np.array_equal(ref2.view(np.uint32), got2.view(np.uint32))
    # call 3: a masked batch again, where a stale tile list would show
    lens3 = np.array([0, 70, 5], dtype=np.int64)
    layers3, mask3 = _case(73, [(512, 256)], 3, 128, 16, lens3)
    say("[noalloc] call 3: masked batch with an empty example")
    ref3, got3, _ = _both(layers3, mask3, 3, 128, 16, P.F32)
    assert np.array_equal(ref3.view(np.uint32), got3.view(np.uint32))
    assert (got3[0, :256] == 0).all()


def test_noalloc_rejects_batches_beyond_its_workspace():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import say
    lib = P.lib()
    B, T, n, k = 1, 40960, 1024, 128
    x = torch.zeros((B, T, n), dtype=torch.bfloat16, device="cuda")
    p = torch.zeros((k, n), dtype=torch.bfloat16, device="cuda")
    g = torch.zeros((B, k * k), dtype=torch.float32, device="cuda")
    arr = (P.LayerDesc * 1)(P.LayerDesc(x.data_ptr(), x.data_ptr(), p.data_ptr(), p.data_ptr(), g.data_ptr(), n, n))
    need = lib.logra_project_layers_ws_size(arr, 1, B, T, k, k)
    say(f"[noalloc] a batch needing {need / 2**20:.1f} MiB")
    assert need > P.NOALLOC_WS_BYTES
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = lib.logra_project_layers_noalloc(arr, 1, P.BF16, B, T, None, k, k, P.F32, k * k, stream)
    assert rc == P.ERR_UNSUPPORTED
    assert "no-allocation" in P.logra_last_error()
    assert lib.logra_project_layers_noalloc(arr, 1, P.BF16, 0, T, None, k, k, P.F32, k * k, stream) == P.OK
    torch.cuda.synchronize()
