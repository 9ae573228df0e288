"""GPU parity of out-of-core scoring: a store in pinned host memory streamed
in chunks through two device staging buffers (Sec. 4.2: the reading of
training gradients overlapped with the influence computation) must give the
exact top-k of the whole store -- bit for bit the oracle's on integer scores,
and bit for bit the device-resident call's on real-valued ones (every score
is the same dot product in the same order wherever its row sits)."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


def _pinned(a):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16) if a.dtype == np.uint16 else np.ascontiguousarray(a))
    if a.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.pin_memory()


def _stream(te, tr_host, k, chunk, copy_stream=None):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    Q = te.shape[0]
    tv = torch.empty((Q, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((Q, k), dtype=torch.int64, device="cuda")
    P.logra_influence_stream(dev(te), tr_host, k, tv, ti, chunk, copy_stream=copy_stream)
    return host(tv), host(ti)


def _resident(te, tr, k):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    Q = te.shape[0]
    tv = torch.empty((Q, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((Q, k), dtype=torch.int64, device="cuda")
    P.logra_influence_scores(dev(te), dev(tr), topk=k, topk_val=tv, topk_idx=ti)
    torch.cuda.synchronize()
    return host(tv), host(ti)


def test_stream_integer_exact_ragged_chunks():
    from gpu_util import say
    say("[stream] integer scores, 24,000 rows in chunks of 7,000 (ragged last)")
    g = W.rng(70)
    Q, N, D, k = 9, 24_000, 64, 37
    te = W.integer_array(g, (Q, D), -2, 2, "bf16", 0.5)
    tr = W.integer_array(g, (N, D), -2, 2, "bf16", 0.5)
    wv, wi = oracle.topk(oracle.scores(te, tr), k)
    tv, ti = _stream(te, _pinned(tr), k, 7_000)
    assert np.array_equal(ti, wi)
    assert np.array_equal(tv.astype(np.float64), wv)


def test_stream_equals_resident_strided_store():
    import torch
    from gpu_util import say
    say("[stream] real scores, host rows at a stride, chunks of 1,500 and of 7")
    g = W.rng(71)
    Q, N, D, ld, k = 20, 5_000, 136, 200, 50
    te = W.normal(g, (Q, D), 1.0, "bf16")
    full = W.normal(g, (N, ld), 1.0, "bf16")
    tr = np.ascontiguousarray(full[:, :D])
    rv, ri = _resident(te, tr, k)
    host_full = _pinned(full)
    tv, ti = _stream(te, host_full[:, :D], k, 1_500)
    assert np.array_equal(ti, ri) and np.array_equal(tv, rv)
    side = torch.cuda.Stream()                       # the caller's copy stream
    tv2, ti2 = _stream(te[:3], _pinned(tr[:50]), 10, 7, copy_stream=side)   # chunks smaller than k
    rv2, ri2 = _resident(te[:3], tr[:50], 10)
    assert np.array_equal(ti2, ri2) and np.array_equal(tv2, rv2)


def test_stream_single_chunk_empty_store_and_pageable_rejected():
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host, say
    say("[stream] one chunk, empty store, pageable memory")
    g = W.rng(72)
    te = W.normal(g, (4, 32), 1.0, "f32")
    tr = W.normal(g, (300, 32), 1.0, "f32")
    tv, ti = _stream(te, _pinned(tr), 8, 1_000)
    rv, ri = _resident(te, tr, 8)
    assert np.array_equal(ti, ri) and np.array_equal(tv, rv)
    tv, ti = _stream(te, _pinned(tr[:0]), 5, 64)
    assert np.all(ti == -1) and np.all(np.isneginf(tv))
    tvd = torch.empty((4, 8), dtype=torch.float32, device="cuda")
    tid = torch.empty((4, 8), dtype=torch.int64, device="cuda")
    with pytest.raises(P.LograError) as ei:
        P.logra_influence_stream(dev(te), torch.from_numpy(tr), 8, tvd, tid, 100)   # pageable
    assert ei.value.status == P.ERR_INVALID_ARG and "pinned" in P.logra_last_error()
