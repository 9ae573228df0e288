// Out-of-core store on disk (the paper's store of projected training
// gradients outgrows host memory too: Table 1 puts it at 3.5 TB; Sec. 4.2
// Efficiency and App. E.2 hide the data IO behind the computation).
//
// A store file holds N rows of row_bytes each, packed, from a byte offset of
// an open file descriptor -- the layout logra_offload_rows_file writes.
//   - logra_store_read_rows / logra_store_write_rows: positioned reads and
//     writes of row ranges (host memory), retried on EINTR and short counts;
//   - logra_influence_stream_file: a reader thread preads chunk c + 1 into one
//     of two pinned host buffers while chunk c is copied to the device and
//     chunk c - 1 is scored, the device side being logra_influence_stream's
//     double buffer;
//   - logra_offload_rows_file: device rows to a pinned host buffer, then a
//     host function enqueued on the same stream writes them to the file, so
//     the caller's thread never waits for the disk.
#include <errno.h>
#include <fcntl.h>
#include <hip/hip_runtime.h>
#include <unistd.h>

#include <condition_variable>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <thread>

#include "internal.h"
#include "logra.h"

namespace {

// Reads or writes `bytes` at `off` in full; 0, or errno (EIO for a read that
// meets the end of the file).
int pread_all(int fd, void *dst, size_t bytes, int64_t off) {
    char *p = static_cast<char *>(dst);
    while (bytes > 0) {
        const ssize_t r = pread(fd, p, bytes, static_cast<off_t>(off));
        if (r < 0) {
            if (errno == EINTR) continue;
            return errno;
        }
        if (r == 0) return EIO;   // end of file before the rows ended
        p += r;
        off += r;
        bytes -= static_cast<size_t>(r);
    }
    return 0;
}

int pwrite_all(int fd, const void *src, size_t bytes, int64_t off) {
    const char *p = static_cast<const char *>(src);
    while (bytes > 0) {
        const ssize_t r = pwrite(fd, p, bytes, static_cast<off_t>(off));
        if (r < 0) {
            if (errno == EINTR) continue;
            return errno;
        }
        p += r;
        off += r;
        bytes -= static_cast<size_t>(r);
    }
    return 0;
}

size_t round256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

}  // namespace

extern "C" {

int logra_store_read_rows(int fd, int64_t file_offset, int64_t row0, int64_t rows, int64_t row_bytes, void *dst,
                          int64_t ld_dst) {
    if (fd < 0 || file_offset < 0 || row0 < 0 || rows < 0 || row_bytes <= 0 || ld_dst < row_bytes)
        return logra::fail_code(LOGRA_ERR_INVALID_ARG, "need fd >= 0, offsets and rows >= 0, 0 < row_bytes <= ld_dst");
    if (rows == 0) return logra::ok_code();
    if (dst == nullptr) return logra::fail_code(LOGRA_ERR_INVALID_ARG, "dst is NULL");
    const int64_t base = file_offset + row0 * row_bytes;
    char *d = static_cast<char *>(dst);
    if (ld_dst == row_bytes) {
        const int e = pread_all(fd, d, static_cast<size_t>(rows * row_bytes), base);
        if (e) return logra::fail_code(LOGRA_ERR_IO, "store read of rows %lld..%lld: %s", (long long)row0,
                                       (long long)(row0 + rows - 1), strerror(e));
        return logra::ok_code();
    }
    for (int64_t r = 0; r < rows; ++r) {
        const int e = pread_all(fd, d + r * ld_dst, static_cast<size_t>(row_bytes), base + r * row_bytes);
        if (e) return logra::fail_code(LOGRA_ERR_IO, "store read of row %lld: %s", (long long)(row0 + r), strerror(e));
    }
    return logra::ok_code();
}

int logra_store_write_rows(int fd, int64_t file_offset, int64_t row0, int64_t rows, int64_t row_bytes,
                           const void *src, int64_t ld_src) {
    if (fd < 0 || file_offset < 0 || row0 < 0 || rows < 0 || row_bytes <= 0 || ld_src < row_bytes)
        return logra::fail_code(LOGRA_ERR_INVALID_ARG, "need fd >= 0, offsets and rows >= 0, 0 < row_bytes <= ld_src");
    if (rows == 0) return logra::ok_code();
    if (src == nullptr) return logra::fail_code(LOGRA_ERR_INVALID_ARG, "src is NULL");
    const int64_t base = file_offset + row0 * row_bytes;
    const char *s = static_cast<const char *>(src);
    if (ld_src == row_bytes) {
        const int e = pwrite_all(fd, s, static_cast<size_t>(rows * row_bytes), base);
        if (e) return logra::fail_code(LOGRA_ERR_IO, "store write: %s", strerror(e));
        return logra::ok_code();
    }
    for (int64_t r = 0; r < rows; ++r) {
        const int e = pwrite_all(fd, s + r * ld_src, static_cast<size_t>(row_bytes), base + r * row_bytes);
        if (e) return logra::fail_code(LOGRA_ERR_IO, "store write of row %lld: %s", (long long)(row0 + r), strerror(e));
    }
    return logra::ok_code();
}

size_t logra_influence_stream_file_ws_size(int Q, int64_t chunk_rows, int D, int tr_dtype, int topk) {
    return logra_influence_stream_ws_size(Q, chunk_rows, D, tr_dtype, topk);
}

int logra_influence_stream_file(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q, int fd, int64_t file_offset,
                                int tr_dtype, int64_t N, int D, int64_t chunk_rows, int topk, float *topk_val,
                                int64_t *topk_idx, void *host_buf, size_t host_buf_bytes, void *ws, size_t ws_bytes,
                                void *stream, void *copy_stream) {
    if (fd < 0 || file_offset < 0) return logra::fail_code(LOGRA_ERR_INVALID_ARG, "need fd >= 0 and file_offset >= 0");
    if (tr_dtype != LOGRA_F32 && tr_dtype != LOGRA_BF16 && tr_dtype != LOGRA_F64)
        return logra::fail_code(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if (Q < 0 || N < 0 || D <= 0 || chunk_rows <= 0 || topk <= 0)
        return logra::fail_code(LOGRA_ERR_INVALID_ARG, "need Q >= 0, N >= 0, D > 0, chunk_rows > 0, topk > 0");
    if ((te_dtype == LOGRA_BF16) != (tr_dtype == LOGRA_BF16))
        return logra::fail_code(LOGRA_ERR_UNSUPPORTED, "bf16 scores need both operands in bf16");
    const size_t es = tr_dtype == LOGRA_BF16 ? 2 : tr_dtype == LOGRA_F64 ? 8 : 4;
    const size_t chunk_bytes = static_cast<size_t>(chunk_rows) * static_cast<size_t>(D) * es;
    if (Q == 0) return logra::ok_code();
    if (N == 0)   // an empty store: top-k padding, through the device-resident path
        return logra_influence_stream(g_test_pre, te_dtype, ld_te, Q, nullptr, tr_dtype, D, 0, D, chunk_rows, topk,
                                      topk_val, topk_idx, ws, ws_bytes, stream, copy_stream);
    if (host_buf == nullptr || host_buf_bytes < 2 * round256(chunk_bytes))
        return logra::fail_code(LOGRA_ERR_WORKSPACE, "host_buf needs %zu bytes of pinned host memory, got %zu",
                                2 * round256(chunk_bytes), host_buf ? host_buf_bytes : size_t{0});
    int rc = logra::check_pinned_code(host_buf, "host_buf", 16);
    if (rc != LOGRA_OK) return rc;
    rc = logra::check_pinned_code(static_cast<char *>(host_buf) + 2 * round256(chunk_bytes) - 1, "the end of host_buf", 1);
    if (rc != LOGRA_OK) return rc;
    // the scoring of each chunk: validate once, on the first chunk's shape
    const size_t need = logra_influence_stream_ws_size(Q, chunk_rows, D, tr_dtype, topk);
    if (ws == nullptr || ws_bytes < need)
        return logra::fail_code(LOGRA_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws ? ws_bytes : size_t{0});
    char *hb[2] = {static_cast<char *>(host_buf), static_cast<char *>(host_buf) + round256(chunk_bytes)};
    const size_t stage = round256(chunk_bytes);
    char *dbuf[2] = {static_cast<char *>(ws), static_cast<char *>(ws) + stage};
    void *iws = static_cast<char *>(ws) + 2 * stage;
    const size_t iws_bytes = ws_bytes - 2 * stage;
    const int64_t chunks = (N + chunk_rows - 1) / chunk_rows;
    const int64_t row_bytes = static_cast<int64_t>(D) * static_cast<int64_t>(es);

    (void)posix_fadvise(fd, static_cast<off_t>(file_offset), static_cast<off_t>(N * row_bytes), POSIX_FADV_SEQUENTIAL);
    // reader thread: chunk c into host buffer c % 2 once that buffer's last
    // copy to the device has completed
    struct Shared {
        std::mutex m;
        std::condition_variable cv;
        int64_t filled[2] = {-1, -1};   // chunk held by each host buffer, -1 = none
        bool free_[2] = {true, true};
        bool stop = false;
        int err = 0;
        int64_t err_chunk = -1;
    } sh;
    std::thread reader([&] {
        for (int64_t c = 0; c < chunks; ++c) {
            const int b = static_cast<int>(c & 1);
            {
                std::unique_lock<std::mutex> lk(sh.m);
                sh.cv.wait(lk, [&] { return sh.free_[b] || sh.stop; });
                if (sh.stop) return;
                sh.free_[b] = false;
            }
            const int64_t r0 = c * chunk_rows, rows = N - r0 < chunk_rows ? N - r0 : chunk_rows;
            const int e = pread_all(fd, hb[b], static_cast<size_t>(rows * row_bytes), file_offset + r0 * row_bytes);
            std::lock_guard<std::mutex> lk(sh.m);
            if (e) {
                sh.err = e;
                sh.err_chunk = c;
                sh.cv.notify_all();
                return;
            }
            sh.filled[b] = c;
            sh.cv.notify_all();
        }
    });

    const hipStream_t cs = static_cast<hipStream_t>(stream);
    hipStream_t xs = static_cast<hipStream_t>(copy_stream);
    const bool own = xs == nullptr;
    hipError_t e = hipSuccess;
    rc = LOGRA_OK;
    if (own && (e = hipStreamCreateWithFlags(&xs, hipStreamNonBlocking)) != hipSuccess) {
        rc = logra::hip_fail(e, "copy stream");
        xs = nullptr;
    }
    hipEvent_t copied[2] = {nullptr, nullptr}, freed[2] = {nullptr, nullptr};
    for (int b = 0; b < 2 && rc == LOGRA_OK; ++b) {
        e = hipEventCreateWithFlags(&copied[b], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&freed[b], hipEventDisableTiming);
        if (e != hipSuccess) rc = logra::hip_fail(e, "event");
    }
    for (int64_t c = 0; c < chunks && rc == LOGRA_OK; ++c) {
        const int b = static_cast<int>(c & 1);
        {
            std::unique_lock<std::mutex> lk(sh.m);
            sh.cv.wait(lk, [&] { return sh.filled[b] == c || sh.err != 0; });
            if (sh.filled[b] != c) {
                rc = logra::fail_code(LOGRA_ERR_IO, "store file read of chunk %lld (rows from %lld): %s",
                                      (long long)sh.err_chunk, (long long)(sh.err_chunk * chunk_rows),
                                      sh.err == EIO ? "the file ends before the store does" : strerror(sh.err));
                break;
            }
        }
        const int64_t r0 = c * chunk_rows, rows = N - r0 < chunk_rows ? N - r0 : chunk_rows;
        if (c >= 2 && (e = hipStreamWaitEvent(xs, freed[b], 0)) != hipSuccess) {
            rc = logra::hip_fail(e, "wait for a free device buffer");
            break;
        }
        e = hipMemcpyAsync(dbuf[b], hb[b], static_cast<size_t>(rows * row_bytes), hipMemcpyHostToDevice, xs);
        if (e == hipSuccess) e = hipEventRecord(copied[b], xs);
        // the host buffer is free for the reader once its copy has completed
        if (e == hipSuccess) e = hipEventSynchronize(copied[b]);
        if (e != hipSuccess) {
            rc = logra::hip_fail(e, "chunk copy");
            break;
        }
        {
            std::lock_guard<std::mutex> lk(sh.m);
            sh.filled[b] = -1;
            sh.free_[b] = true;
            sh.cv.notify_all();
        }
        if ((e = hipStreamWaitEvent(cs, copied[b], 0)) != hipSuccess) {
            rc = logra::hip_fail(e, "order the scoring after the copy");
            break;
        }
        rc = logra_influence_scores(g_test_pre, te_dtype, ld_te, Q, dbuf[b], tr_dtype, D, rows, D, r0, nullptr, 1,
                                    topk, topk_val, topk_idx, c > 0, iws, iws_bytes, stream);
        if (rc == LOGRA_OK && (e = hipEventRecord(freed[b], cs)) != hipSuccess) rc = logra::hip_fail(e, "event record");
    }
    {
        std::lock_guard<std::mutex> lk(sh.m);
        sh.stop = true;
        sh.cv.notify_all();
    }
    reader.join();
    e = hipStreamSynchronize(cs);
    if (rc == LOGRA_OK && e != hipSuccess) rc = logra::hip_fail(e, "stream synchronize");
    if (xs) {
        e = hipStreamSynchronize(xs);
        if (rc == LOGRA_OK && e != hipSuccess) rc = logra::hip_fail(e, "copy stream synchronize");
    }
    for (int b = 0; b < 2; ++b) {
        if (copied[b]) (void)hipEventDestroy(copied[b]);
        if (freed[b]) (void)hipEventDestroy(freed[b]);
    }
    if (own && xs) (void)hipStreamDestroy(xs);
    return rc == LOGRA_OK ? logra::ok_code() : rc;
}

namespace {
struct WriteJob {
    int fd;
    int64_t offset;
    const void *buf;
    size_t bytes;
    int *status;
};
// Runs on a runtime thread once the copy before it on the stream has
// completed; calls no HIP function.
void write_job(void *p) {
    WriteJob *j = static_cast<WriteJob *>(p);
    const int e = pwrite_all(j->fd, j->buf, j->bytes, j->offset);
    if (j->status) *j->status = e ? LOGRA_ERR_IO : LOGRA_OK;
    delete j;
}
}  // namespace

int logra_offload_rows_file(const void *src, int64_t ld_src, int64_t rows, int64_t row_bytes, int fd,
                            int64_t file_offset, void *host_buf, size_t host_buf_bytes, int *io_status, void *stream,
                            void *copy_stream, void *done) {
    if (rows < 0 || row_bytes <= 0 || ld_src < row_bytes || fd < 0 || file_offset < 0)
        return logra::fail_code(LOGRA_ERR_INVALID_ARG,
                                "need rows >= 0, 0 < row_bytes <= ld_src, fd >= 0 and file_offset >= 0");
    if (rows == 0) {
        if (io_status) *io_status = LOGRA_OK;
        return logra::ok_code();
    }
    const size_t bytes = static_cast<size_t>(rows * row_bytes);
    if (host_buf == nullptr || host_buf_bytes < bytes)
        return logra::fail_code(LOGRA_ERR_WORKSPACE, "host_buf needs %zu bytes of pinned host memory", bytes);
    // device rows to the packed pinned buffer (same checks and ordering as logra_offload_rows)
    int rc = logra_offload_rows(src, ld_src, host_buf, row_bytes, rows, row_bytes, stream, copy_stream, nullptr);
    if (rc != LOGRA_OK) return rc;
    const hipStream_t xs = static_cast<hipStream_t>(copy_stream ? copy_stream : stream);
    if (io_status) *io_status = 1;   // pending
    WriteJob *job = new WriteJob{fd, file_offset, host_buf, bytes, io_status};
    hipError_t e = hipLaunchHostFunc(xs, write_job, job);
    if (e != hipSuccess) {
        delete job;
        return logra::hip_fail(e, "enqueue the file write");
    }
    if (done && (e = hipEventRecord(static_cast<hipEvent_t>(done), xs)) != hipSuccess)
        return logra::hip_fail(e, "record done");
    return logra::ok_code();
}

}  // extern "C"
