"""GPU parity of the disk tier of the out-of-core store (Sec. 4.2 Efficiency,
App. E.2; Table 1's store outgrows host memory): store rows written from the
device with logra_offload_rows_file land in the file bit for bit, and
logra_influence_stream_file over that file gives the exact top-k of the
whole store -- the oracle's on integer scores, the device-resident call's bit
for bit on real ones.  A file that ends early is reported as an IO error."""
import ctypes
import os
import tempfile

import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture
def path():
    f = tempfile.NamedTemporaryFile(prefix="logra_store_", delete=False)
    f.close()
    yield f.name
    os.unlink(f.name)


def _pinned_bytes(n):
    import torch
    return torch.empty(max(n, 1), dtype=torch.uint8).pin_memory()


def _write_store(path, tr_dev, batch):
    """The rows of the device store written batch by batch with write-behind; returns io statuses."""
    import torch
    import paper_2405_13954_amd as P
    fd = os.open(path, os.O_RDWR | os.O_TRUNC)
    try:
        rb = tr_dev.shape[1] * tr_dev.element_size()
        bufs = [_pinned_bytes(batch * rb) for _ in range(2)]
        stats, events = [], []
        for i, r0 in enumerate(range(0, tr_dev.shape[0], batch)):
            if i >= 2:
                events[i - 2].synchronize()          # that buffer's write has run
            st, ev = ctypes.c_int(-7), torch.cuda.Event()
            P.logra_offload_rows_file(tr_dev[r0:r0 + batch], fd, r0 * rb, bufs[i % 2], io_status=st, done=ev)
            stats.append(st)
            events.append(ev)
        torch.cuda.synchronize()
        return [s.value for s in stats]
    finally:
        os.close(fd)


def _stream_file(path, te, N, D, dtype_code, k, chunk):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import dev, host
    Q = te.shape[0]
    es = {P.BF16: 2, P.F32: 4, P.F64: 8}[dtype_code]
    tv = torch.empty((Q, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((Q, k), dtype=torch.int64, device="cuda")
    hb = _pinned_bytes(2 * ((chunk * D * es + 255) // 256 * 256))
    fd = os.open(path, os.O_RDONLY)
    try:
        P.logra_influence_stream_file(dev(te), fd, 0, N, D, dtype_code, k, tv, ti, chunk, hb)
    finally:
        os.close(fd)
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


def test_offload_to_file_then_stream_integer_exact(path):
    import paper_2405_13954_amd as P
    from gpu_util import dev, say
    say("[store file] 24,000 integer rows written from the device in batches of 2,500, streamed in chunks of 7,000")
    g = W.rng(90)
    Q, N, D, k = 9, 24_000, 64, 37
    te = W.integer_array(g, (Q, D), -2, 2, "bf16", 0.5)
    tr = W.integer_array(g, (N, D), -2, 2, "bf16", 0.5)
    stats = _write_store(path, dev(tr), 2_500)
    assert all(s == P.OK for s in stats)
    on_disk = np.fromfile(path, dtype=np.uint16).reshape(N, D)
    assert np.array_equal(on_disk, tr)
    wv, wi = oracle.topk(oracle.scores(te, tr), k)
    tv, ti = _stream_file(path, te, N, D, P.BF16, k, 7_000)
    assert np.array_equal(ti, wi) and np.array_equal(tv.astype(np.float64), wv)


def test_stream_file_equals_resident_from_disk(path):
    import paper_2405_13954_amd as P
    from gpu_util import say
    say("[store file] real scores, 6,000 rows of 2,048 bf16, chunks of 1,000; page cache, then evicted")
    g = W.rng(91)
    Q, N, D, k = 12, 6_000, 2048, 40
    te = W.normal(g, (Q, D), 1.0, "bf16")
    tr = W.normal(g, (N, D), 1.0, "bf16")
    tr.tofile(path)
    rv, ri = _resident(te, tr, k)
    tv, ti = _stream_file(path, te, N, D, P.BF16, k, 1_000)
    assert np.array_equal(ti, ri) and np.array_equal(tv, rv)
    fd = os.open(path, os.O_RDONLY)             # evict the file's pages: the next pass reads the disk
    os.fsync(fd)
    os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
    os.close(fd)
    tv2, ti2 = _stream_file(path, te, N, D, P.BF16, k, 1_000)
    assert np.array_equal(ti2, ri) and np.array_equal(tv2, rv)


def test_stream_file_short_file_is_an_io_error(path):
    import torch
    import paper_2405_13954_amd as P
    from gpu_util import say
    say("[store file] a file that ends before the store does")
    g = W.rng(92)
    te = W.normal(g, (3, 32), 1.0, "f32")
    tr = W.normal(g, (500, 32), 1.0, "f32")
    tr[:450].tofile(path)
    with pytest.raises(P.LograError) as ei:
        _stream_file(path, te, 500, 32, P.F32, 5, 100)
    assert ei.value.status == P.ERR_IO and "ends before" in P.logra_last_error()
    torch.cuda.synchronize()
    tv, ti = _stream_file(path, te[:, :], 450, 32, P.F32, 5, 100)    # the rows that are there
    rv, ri = _resident(te, tr[:450], 5)
    assert np.array_equal(ti, ri) and np.array_equal(tv, rv)
