"""The whole Llama3-8B logging stream at its full size (Sec. 3.1 Eq. (5) and
Sec. 2 Eq. (3) over a complete logging run): 65,536 examples in 8,192
batches of B=8 (T=2048, lengths U{128..2048}), every batch through all 224
layers (8 grouped launches of 28 layers, four blocks each, k=16, as the
bench runs them) into the bf16 store of
65,536 rows of 57,344, and the 224 covariances (kept as lower triangles)
accumulated over all 65,536 examples.

x / dy are four device buffer sets cycled over the 32 blocks (drawing 2.7 GB
per block and batch would be the whole test); the valid lengths, and so the
masks, differ per batch.  Checks against the float64 oracle: sampled store
rows (first, middle and last batch; first and last example; three layers)
and two covariance blocks over all 65,536 rows.  Every store row is finite
and no entry above a covariance diagonal is touched.  About a minute of
GPU time."""
import ctypes
import time

import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


def test_full_logging_stream():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import host, normwise, say
    w = W.WORKLOADS["llama3_8b_stream"]
    B, T, k = w.B, w.T, w.k_in
    D = k * k
    nlb = len(w.layers)
    n_layers = w.n_layers
    D_tot = n_layers * D
    n_ex = w.extra["examples"]
    n_steps = n_ex // B
    n_buf = 4       # x / dy buffer sets: the four blocks of a launch have their own
    gb = 4          # blocks per grouped launch
    say(f"[full stream] {n_ex} examples in {n_steps} batches of {B}, {n_layers} layers, store {n_ex} x {D_tot} bf16")
    gen = W.torch_generator(0, 600)
    bufs = []
    for _ in range(n_buf):
        st = []
        for _, ni, no in w.layers:
            x = torch.empty((B, T, ni), dtype=torch.bfloat16, device="cuda")
            dy = torch.empty((B, T, no), dtype=torch.bfloat16, device="cuda")
            W.device_normal_(x, w.x_std, gen)
            W.device_normal_(dy, w.dy_std, gen)
            st.append((x, dy))
        bufs.append(st)
    projs = []
    for l in range(n_layers):
        _, ni, no = w.layers[l % nlb]
        pi = torch.empty((k, ni), dtype=torch.bfloat16, device="cuda")
        po = torch.empty((k, no), dtype=torch.bfloat16, device="cuda")
        W.device_normal_(pi, 1.0 / np.sqrt(k), gen)
        W.device_normal_(po, 1.0 / np.sqrt(k), gen)
        projs.append((pi, po))
    store = torch.empty((n_ex, D_tot), dtype=torch.bfloat16, device="cuda")
    S = torch.triu(torch.full((n_layers, D, D), float("nan"), dtype=torch.float32, device="cuda"), 1)
    lens = [W.lengths(W.rng(0, 610, s), B, w.len_lo, w.len_hi) for s in range(n_steps)]
    masks = torch.from_numpy(np.stack([W.mask_from_lengths(L_, T) for L_ in lens])).cuda()
    L = P.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    nll = gb * nlb
    shape = (P.LayerDesc * nll)(*[P.LayerDesc(0, 0, 0, 0, 0, ni, no) for _ in range(gb) for _, ni, no in w.layers])
    wsb = P.logra_project_layers_ws_size(shape, nll, B, T, k, k)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    g_ld = store.stride(0)
    row_bytes = g_ld * 2
    # one descriptor array per launch; only the store rows change from batch to batch
    descs = []
    for li in range(n_layers // nll):
        arr = (P.LayerDesc * nll)()
        for bb in range(gb):
            blk = li * gb + bb
            for j, (_, ni, no) in enumerate(w.layers):
                x, dy = bufs[blk % n_buf][j]
                pi, po = projs[blk * nlb + j]
                arr[bb * nlb + j] = P.LayerDesc(x.data_ptr(), dy.data_ptr(), pi.data_ptr(), po.data_ptr(),
                                                store[0:1, (blk * nlb + j) * D:].data_ptr(), ni, no)
        descs.append(arr)
    g0 = [[arr[j].g_out for j in range(nll)] for arr in descs]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(n_steps):
        mp = ctypes.c_void_p(masks[s].data_ptr())
        for li, arr in enumerate(descs):
            for j in range(nll):
                arr[j].g_out = g0[li][j] + s * B * row_bytes
            rc = L.logra_project_layers(arr, nll, P.BF16, B, T, mp, k, k, P.BF16, g_ld,
                                        ctypes.c_void_p(ws.data_ptr()), wsb, stream)
            assert rc == 0, P.logra_last_error()
        rc = L.logra_cov_accumulate_blocks_lower(ctypes.c_void_p(store[s * B].data_ptr()), P.BF16, g_ld, B, D,
                                                 n_layers, ctypes.c_void_p(S.data_ptr()), stream)
        assert rc == 0, P.logra_last_error()
        if s % 1024 == 1023:
            torch.cuda.synchronize()
            say(f"  {s + 1} batches, {time.perf_counter() - t0:.1f} s")
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    tokens = int(sum(int(L_.sum()) for L_ in lens))
    say(f"  {tokens} valid tokens in {dt:.1f} s = {tokens / dt:.3e} tokens/s (projection and covariance)")
    assert bool(torch.isfinite(store).all())
    up = np.triu(np.ones((D, D), bool), 1)
    # sampled store rows: three batches, the first and last example, three layers
    for l in (0, 115, 223):
        blk, j = divmod(l, nlb)
        x, dy = bufs[blk % n_buf][j]
        pi, po = projs[l]
        xh, dyh = host(x[[0, B - 1]]), host(dy[[0, B - 1]])
        pih, poh = host(pi), host(po)
        for s in (0, n_steps // 2, n_steps - 1):
            m = W.mask_from_lengths(lens[s], T)[[0, B - 1]]
            want = oracle.project_factored(xh, dyh, pih, poh, m)
            got = host(store[[s * B, s * B + B - 1], l * D:(l + 1) * D])
            err = max(normwise(got[i], want[i]) for i in range(2))
            say(f"  layer {l}, batch {s}: max normwise err {err:.2e}")
            assert err <= 2e-2
    # two covariance blocks over all 65,536 rows
    for l in (0, 223):
        got = host(S[l])
        assert np.all(np.isnan(got[up]))
        full = np.where(up, got.T, got).astype(np.float64)
        want = oracle.cov_accumulate(host(store[:, l * D:(l + 1) * D]))
        err = normwise(full, want)
        say(f"  covariance of layer {l} over {n_ex} rows: normwise err {err:.2e}")
        assert err <= 1e-4
