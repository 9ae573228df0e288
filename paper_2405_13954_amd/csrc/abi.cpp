// C ABI of the LoGra hot path: argument validation, workspace carving and
// dispatch to the HIP kernels.  Size, dtype and limit checks run before any
// HIP call; pointer checks follow (hipPointerGetAttributes); then launches.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <vector>

#include "internal.h"
#include "logra.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_err[0] = '\0';
    return LOGRA_OK;
}

// Storage types of activations, gradients and stores; fp64 is accepted where
// a call documents it (fp64 statistics of fp32 workloads).
bool valid_dtype(int d) { return d == LOGRA_F32 || d == LOGRA_BF16; }
bool valid_dtype64(int d) { return valid_dtype(d) || d == LOGRA_F64; }
size_t esize(int d) { return d == LOGRA_BF16 ? 2 : d == LOGRA_F64 ? 8 : 4; }
// A score pair: both bf16 (bf16 MFMA), or any mix of fp32 and fp64 (float64
// accumulation).
int check_score_dtypes(int te_dtype, int tr_dtype) {
    if (!valid_dtype64(te_dtype) || !valid_dtype64(tr_dtype)) return fail(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if ((te_dtype == LOGRA_BF16) != (tr_dtype == LOGRA_BF16))
        return fail(LOGRA_ERR_UNSUPPORTED, "bf16 scores need both operands in bf16");
    return LOGRA_OK;
}
bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Device-memory check; `align` is the required base alignment in bytes.
int check_dev(const void *p, const char *name, size_t align) {
    if (p == nullptr) return fail(LOGRA_ERR_INVALID_ARG, "%s is NULL", name);
    if ((reinterpret_cast<uintptr_t>(p) & (align - 1)) != 0)
        return fail(LOGRA_ERR_INVALID_ARG, "%s is not %zu-byte aligned", name, align);
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof attr);
    const hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(LOGRA_ERR_INVALID_ARG, "%s is not device memory (%s)", name, hipGetErrorString(e));
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
        return fail(LOGRA_ERR_INVALID_ARG, "%s is not device memory", name);
    return LOGRA_OK;
}

// Pinned (page-locked) host memory, which asynchronous copies need.
int check_pinned(const void *p, const char *name, size_t align) {
    if (p == nullptr) return fail(LOGRA_ERR_INVALID_ARG, "%s is NULL", name);
    if ((reinterpret_cast<uintptr_t>(p) & (align - 1)) != 0)
        return fail(LOGRA_ERR_INVALID_ARG, "%s is not %zu-byte aligned", name, align);
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof attr);
    const hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess || attr.type != hipMemoryTypeHost) {
        (void)hipGetLastError();
        return fail(LOGRA_ERR_INVALID_ARG, "%s is not pinned host memory (allocate it with hipHostMalloc)", name);
    }
    return LOGRA_OK;
}

}  // namespace

int logra::check_pinned_code(const void *p, const char *name, size_t align) { return check_pinned(p, name, align); }

int logra::hip_fail(hipError_t e, const char *what) {
    return fail(LOGRA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}
int logra::fail_unsupported(const char *msg) { return fail(LOGRA_ERR_UNSUPPORTED, "%s", msg); }
int logra::fail_code(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}
int logra::ok_code() { return ok(); }

namespace {
using logra::hip_fail;

#define TRY(expr)                       \
    do {                                \
        const int rc_ = (expr);         \
        if (rc_ != LOGRA_OK) return rc_; \
    } while (0)

int check_ws(void *ws, size_t ws_bytes, size_t need) {
    if (need == 0) return LOGRA_OK;
    if (ws == nullptr || ws_bytes < need)
        return fail(LOGRA_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws ? ws_bytes : 0);
    return check_dev(ws, "ws", 256);
}

size_t round256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

int check_proj_sizes(int in_dtype, int B, int T, int n_in, int n_out, int k_in, int k_out,
                     int g_dtype, int64_t g_ld) {
    if (!valid_dtype(in_dtype) || !valid_dtype(g_dtype)) return fail(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if (B < 0 || T < 0) return fail(LOGRA_ERR_INVALID_ARG, "B and T must be >= 0");
    if (n_in <= 0 || n_out <= 0 || k_in <= 0 || k_out <= 0)
        return fail(LOGRA_ERR_INVALID_ARG, "n_in, n_out, k_in, k_out must be > 0");
    const int vec = in_dtype == LOGRA_BF16 ? 8 : 4;
    if (n_in % vec || n_out % vec)
        return fail(LOGRA_ERR_INVALID_ARG, "n_in and n_out must be multiples of %d", vec);
    if (k_in > LOGRA_MAX_K || k_out > LOGRA_MAX_K)
        return fail(LOGRA_ERR_UNSUPPORTED, "k_in, k_out must be <= %d", LOGRA_MAX_K);
    if (g_ld < static_cast<int64_t>(k_in) * k_out)
        return fail(LOGRA_ERR_INVALID_ARG, "g_ld must be >= k_in * k_out");
    if (static_cast<int64_t>(B) * T * (n_in > n_out ? n_in : n_out) < 0)
        return fail(LOGRA_ERR_INVALID_ARG, "size overflow");
    return LOGRA_OK;
}

}  // namespace

extern "C" {

const char *logra_last_error(void) { return g_err; }
const char *logra_version(void) { return "logra-mi355x 0.1.0 (gfx950)"; }

size_t logra_project_ws_size(int B, int T, int n_in, int n_out, int k_in, int k_out) {
    if (B <= 0 || T <= 0 || n_in <= 0 || n_out <= 0 || k_in <= 0 || k_out <= 0) return 0;
    return round256(logra::project_ws_bytes(&n_in, &n_out, 1, B, T, k_in, k_out));
}

size_t logra_project_layers_ws_size(const logra_layer_desc *layers, int n_layers, int B, int T,
                                    int k_in, int k_out) {
    if (layers == nullptr || n_layers <= 0 || n_layers > LOGRA_MAX_GROUP || B <= 0 || T <= 0 ||
        k_in <= 0 || k_out <= 0)
        return 0;
    int n_in[LOGRA_MAX_GROUP], n_out[LOGRA_MAX_GROUP];
    for (int l = 0; l < n_layers; ++l) {
        if (layers[l].n_in <= 0 || layers[l].n_out <= 0) return 0;
        n_in[l] = layers[l].n_in;
        n_out[l] = layers[l].n_out;
    }
    return round256(logra::project_ws_bytes(n_in, n_out, n_layers, B, T, k_in, k_out));
}

}  // extern "C"

// logra_project_layers; `ws_known` marks a workspace the library owns (the
// no-allocation entry point's static device array), whose pointer kind needs
// no check.
int logra::project_layers_checked(const logra_layer_desc *layers, int n_layers, int in_dtype, int B, int T,
                                  const uint8_t *mask, int k_in, int k_out, int g_dtype, int64_t g_ld, void *ws,
                                  size_t ws_bytes, bool ws_known, void *stream) {
    if (layers == nullptr) return fail(LOGRA_ERR_INVALID_ARG, "layers is NULL");
    if (n_layers < 1 || n_layers > LOGRA_MAX_GROUP)
        return fail(n_layers > LOGRA_MAX_GROUP ? LOGRA_ERR_UNSUPPORTED : LOGRA_ERR_INVALID_ARG,
                    "n_layers must be in 1..%d", LOGRA_MAX_GROUP);
    for (int l = 0; l < n_layers; ++l)
        TRY(check_proj_sizes(in_dtype, B, T, layers[l].n_in, layers[l].n_out, k_in, k_out, g_dtype, g_ld));
    if (B == 0 || T == 0) return ok();
    logra::ProjGroup grp;
    std::memset(&grp, 0, sizeof grp);
    grp.n_layers = n_layers;
    for (int l = 0; l < n_layers; ++l) {
        const logra_layer_desc &d = layers[l];
        TRY(check_dev(d.x, "x", 16));
        TRY(check_dev(d.dy, "dy", 16));
        TRY(check_dev(d.p_in, "p_in", 16));
        TRY(check_dev(d.p_out, "p_out", 16));
        TRY(check_dev(d.g_out, "g_out", esize(g_dtype)));
        // the last element written must lie in device memory too (a wrong row
        // stride is reported instead of faulting the kernel)
        const double span = (static_cast<double>(B - 1) * static_cast<double>(g_ld) + k_in * k_out) *
                            static_cast<double>(esize(g_dtype));
        if (span > 281474976710656.0)   // 2^48 bytes: beyond any device allocation
            return fail(LOGRA_ERR_INVALID_ARG, "g_out rows at stride g_ld = %lld exceed device memory",
                        static_cast<long long>(g_ld));
        const char *g_end = static_cast<const char *>(d.g_out) +
                            (static_cast<int64_t>(B - 1) * g_ld + static_cast<int64_t>(k_in) * k_out - 1) *
                                static_cast<int64_t>(esize(g_dtype));
        TRY(check_dev(g_end, "the last row of g_out", 1));
        grp.layer[l] = {d.x, d.dy, d.p_in, d.p_out, d.g_out, d.n_in, d.n_out};
    }
    if (mask) TRY(check_dev(mask, "mask", 1));
    const size_t need = logra_project_layers_ws_size(layers, n_layers, B, T, k_in, k_out);
    if (ws_known) {
        if (ws_bytes < need)
            return fail(LOGRA_ERR_UNSUPPORTED, "the batch needs %zu bytes of workspace, more than the %zu of the "
                        "no-allocation entry point", need, ws_bytes);
    } else {
        TRY(check_ws(ws, ws_bytes, need));
    }
    const hipError_t e = logra::launch_project(grp, in_dtype == LOGRA_BF16, B, T, mask, k_in, k_out,
                                               g_dtype == LOGRA_BF16, g_ld, ws,
                                               static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "projection launch");
    return ok();
}

extern "C" {

int logra_project_layers(const logra_layer_desc *layers, int n_layers, int in_dtype, int B, int T,
                         const uint8_t *mask, int k_in, int k_out, int g_dtype, int64_t g_ld,
                         void *ws, size_t ws_bytes, void *stream) {
    return logra::project_layers_checked(layers, n_layers, in_dtype, B, T, mask, k_in, k_out, g_dtype, g_ld, ws,
                                         ws_bytes, false, stream);
}

int logra_project_layer(const void *x, const void *dy, int in_dtype, int B, int T, int n_in,
                        int n_out, const uint8_t *mask, const void *p_in, const void *p_out,
                        int k_in, int k_out, void *g_out, int g_dtype, int64_t g_ld, void *ws,
                        size_t ws_bytes, void *stream) {
    logra_layer_desc d;
    d.x = x;
    d.dy = dy;
    d.p_in = p_in;
    d.p_out = p_out;
    d.g_out = g_out;
    d.n_in = n_in;
    d.n_out = n_out;
    return logra_project_layers(&d, 1, in_dtype, B, T, mask, k_in, k_out, g_dtype, g_ld, ws, ws_bytes,
                                stream);
}

static int cov_blocks_impl(const void *g, int g_dtype, int64_t ld, int B, int D, int n_blocks, float *S, bool lower,
                           void *stream) {
    if (!valid_dtype(g_dtype)) return fail(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if (B < 0 || D <= 0 || n_blocks <= 0) return fail(LOGRA_ERR_INVALID_ARG, "need B >= 0, D > 0, n_blocks > 0");
    if (n_blocks > 65535) return fail(LOGRA_ERR_UNSUPPORTED, "n_blocks must be <= 65535");
    if (ld < static_cast<int64_t>(D) * n_blocks) return fail(LOGRA_ERR_INVALID_ARG, "ld must be >= D * n_blocks");
    if (g_dtype == LOGRA_BF16 && (D % 8 || ld % 8))
        return fail(LOGRA_ERR_INVALID_ARG, "bf16 covariance needs D and ld multiples of 8");
    if (B == 0) return ok();
    TRY(check_dev(g, "g", g_dtype == LOGRA_BF16 ? 16 : 4));
    TRY(check_dev(S, "S", 4));
    const hipError_t e = logra::launch_cov(g, g_dtype == LOGRA_BF16, ld, B, D, n_blocks, S, lower,
                                           static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "covariance launch");
    return ok();
}

int logra_cov_accumulate_blocks(const void *g, int g_dtype, int64_t ld, int B, int D, int n_blocks,
                                float *S, void *stream) {
    return cov_blocks_impl(g, g_dtype, ld, B, D, n_blocks, S, false, stream);
}

int logra_cov_accumulate_blocks_lower(const void *g, int g_dtype, int64_t ld, int B, int D, int n_blocks,
                                      float *S, void *stream) {
    return cov_blocks_impl(g, g_dtype, ld, B, D, n_blocks, S, true, stream);
}

int logra_cov_accumulate(const void *g, int g_dtype, int64_t ld, int B, int D, float *S, void *stream) {
    return logra_cov_accumulate_blocks(g, g_dtype, ld, B, D, 1, S, stream);
}

int logra_cov_accumulate_f64(const void *g, int g_dtype, int64_t ld, int B, int D, int n_blocks, double *S,
                             void *stream) {
    if (g_dtype != LOGRA_F32 && g_dtype != LOGRA_F64)
        return fail(LOGRA_ERR_INVALID_ARG, "fp64 covariance takes fp32 or fp64 rows");
    if (B < 0 || D <= 0 || n_blocks <= 0) return fail(LOGRA_ERR_INVALID_ARG, "need B >= 0, D > 0, n_blocks > 0");
    if (n_blocks > 65535) return fail(LOGRA_ERR_UNSUPPORTED, "n_blocks must be <= 65535");
    if (ld < static_cast<int64_t>(D) * n_blocks) return fail(LOGRA_ERR_INVALID_ARG, "ld must be >= D * n_blocks");
    if (B == 0) return ok();
    TRY(check_dev(g, "g", esize(g_dtype)));
    TRY(check_dev(S, "S", 8));
    const hipError_t e = logra::launch_cov_f64(g, g_dtype == LOGRA_F64, ld, B, D, n_blocks, S,
                                               static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "covariance launch");
    return ok();
}

// Waits for `s`, then returns NOT_PD naming the first block whose
// factorisation met a non-positive pivot (the status words in the workspace).
static int report_not_pd(void *ws, int D, int n_blocks, hipStream_t s) {
    std::vector<int> info(static_cast<size_t>(n_blocks), 0);
    hipError_t e = hipMemcpyAsync(info.data(), logra::precond_info_ptr(ws, D, n_blocks), sizeof(int) * n_blocks,
                                  hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return hip_fail(e, "status copy");
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "stream synchronize");
    for (int b = 0; b < n_blocks; ++b)
        if (info[b] != 0)
            return fail(LOGRA_ERR_NOT_PD, "block %d: pivot %d of C + lambda I is not positive", b, info[b] - 1);
    return ok();
}

size_t logra_precondition_ws_size(int D, int n_blocks, int Q) {
    if (D <= 0 || n_blocks <= 0 || Q < 0) return 0;
    return round256(logra::precond_ws_bytes(D, n_blocks, Q));
}

static int precondition_impl(const void *S, bool s_f64, int D, int n_blocks, int64_t N, double damp_ratio,
                             const void *g_test, int in_dtype, int64_t ld_in, int Q, void *g_out, int out_dtype,
                             int64_t ld_out, void *ws, size_t ws_bytes, void *stream) {
    if (!valid_dtype64(in_dtype) || !valid_dtype64(out_dtype)) return fail(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if (D <= 0 || n_blocks <= 0 || Q < 0) return fail(LOGRA_ERR_INVALID_ARG, "need D > 0, n_blocks > 0, Q >= 0");
    if (D > LOGRA_MAX_PRECOND_D) return fail(LOGRA_ERR_UNSUPPORTED, "D must be <= %d", LOGRA_MAX_PRECOND_D);
    if (n_blocks > 65535) return fail(LOGRA_ERR_UNSUPPORTED, "n_blocks must be <= 65535");
    const int64_t width = static_cast<int64_t>(D) * n_blocks;
    if (ld_in < width || ld_out < width) return fail(LOGRA_ERR_INVALID_ARG, "ld_in and ld_out must be >= D * n_blocks");
    if (damp_ratio >= 0.0 && N <= 0) return fail(LOGRA_ERR_INVALID_ARG, "N must be > 0");
    if (damp_ratio != damp_ratio) return fail(LOGRA_ERR_INVALID_ARG, "damp_ratio is NaN");
    if (Q == 0 && damp_ratio < 0.0) return ok();
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (Q > 0) {
        TRY(check_dev(g_test, "g_test", esize(in_dtype)));
        TRY(check_dev(g_out, "g_out", esize(out_dtype)));
    }
    if (damp_ratio < 0.0) {
        hipError_t e = logra::launch_copy_rows(g_test, in_dtype, ld_in, Q, static_cast<int>(width), g_out, out_dtype,
                                               ld_out, s);
        if (e != hipSuccess) return hip_fail(e, "copy launch");
        e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_fail(e, "stream synchronize");
        return ok();
    }
    TRY(check_dev(S, "S", s_f64 ? 8 : 4));
    TRY(check_ws(ws, ws_bytes, logra_precondition_ws_size(D, n_blocks, Q)));
    hipError_t e = logra::launch_precondition(S, s_f64, D, n_blocks, N, damp_ratio, g_test, in_dtype, ld_in, Q,
                                              g_out, out_dtype, ld_out, ws, s);
    if (e != hipSuccess) return hip_fail(e, "precondition launch");
    return report_not_pd(ws, D, n_blocks, s);
}

int logra_precondition_blocks(const float *S, int D, int n_blocks, int64_t N, double damp_ratio,
                              const void *g_test, int in_dtype, int64_t ld_in, int Q, void *g_out,
                              int out_dtype, int64_t ld_out, void *ws, size_t ws_bytes,
                              void *stream) {
    return precondition_impl(S, false, D, n_blocks, N, damp_ratio, g_test, in_dtype, ld_in, Q, g_out, out_dtype,
                             ld_out, ws, ws_bytes, stream);
}

int logra_precondition_f64(const double *S, int D, int n_blocks, int64_t N, double damp_ratio, const void *g_test,
                           int in_dtype, int64_t ld_in, int Q, void *g_out, int out_dtype, int64_t ld_out, void *ws,
                           size_t ws_bytes, void *stream) {
    return precondition_impl(S, true, D, n_blocks, N, damp_ratio, g_test, in_dtype, ld_in, Q, g_out, out_dtype,
                             ld_out, ws, ws_bytes, stream);
}

int logra_precondition(const float *S, int D, int64_t N, double damp_ratio, const void *g_test,
                       int in_dtype, int64_t ld_in, int Q, void *g_out, int out_dtype, int64_t ld_out,
                       void *ws, size_t ws_bytes, void *stream) {
    return logra_precondition_blocks(S, D, 1, N, damp_ratio, g_test, in_dtype, ld_in, Q, g_out, out_dtype,
                                     ld_out, ws, ws_bytes, stream);
}

size_t logra_influence_ws_size(int Q, int64_t N_chunk, int topk, int scores_given) {
    if (Q <= 0 || N_chunk <= 0 || topk <= 0 || topk > LOGRA_MAX_TOPK) return 0;
    const size_t q = static_cast<size_t>(Q);
    size_t b = scores_given ? 0 : round256(sizeof(float) * q * static_cast<size_t>(N_chunk));
    if (logra::topk_prefix_rows(N_chunk, topk) > 0)   // thresholds, counts, candidate lists
        b += 2 * round256(4 * q) + 2 * round256(4 * q * logra::kCandCap);
    return b;
}

static int influence_impl(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q, const void *g_train,
                          int tr_dtype, int64_t ld_tr, int64_t N_chunk, int D, int64_t train_base,
                          float *scores, int64_t ld_s, int topk, float *topk_val, int64_t *topk_idx, int merge,
                          const float *row_scale, const float *col_scale, void *ws, size_t ws_bytes,
                          void *stream) {
    TRY(check_score_dtypes(te_dtype, tr_dtype));
    if (Q < 0 || N_chunk < 0 || D <= 0) return fail(LOGRA_ERR_INVALID_ARG, "need Q >= 0, N_chunk >= 0, D > 0");
    if (ld_te < D || ld_tr < D) return fail(LOGRA_ERR_INVALID_ARG, "ld_te and ld_tr must be >= D");
    if (topk < 0 || topk > LOGRA_MAX_TOPK) return fail(topk < 0 ? LOGRA_ERR_INVALID_ARG : LOGRA_ERR_UNSUPPORTED,
                                                     "topk must be in 0..%d", LOGRA_MAX_TOPK);
    if (scores == nullptr && topk == 0) return fail(LOGRA_ERR_INVALID_ARG, "nothing to compute: scores is NULL and topk is 0");
    if (scores != nullptr && ld_s < N_chunk) return fail(LOGRA_ERR_INVALID_ARG, "ld_s must be >= N_chunk");
    if (train_base < 0) return fail(LOGRA_ERR_INVALID_ARG, "train_base must be >= 0");
    if (N_chunk > INT32_MAX) return fail(LOGRA_ERR_UNSUPPORTED, "N_chunk must be < 2^31");
    if (merge != 0 && merge != 1) return fail(LOGRA_ERR_INVALID_ARG, "merge must be 0 or 1");
    const bool bf16 = te_dtype == LOGRA_BF16;
    if (bf16 && (D % 8 || ld_te % 8 || ld_tr % 8))
        return fail(LOGRA_ERR_INVALID_ARG, "bf16 scores need D, ld_te, ld_tr multiples of 8");
    if (bf16 && (ld_te >= (int64_t{1} << 22) || ld_tr >= (int64_t{1} << 22)))
        return fail(LOGRA_ERR_UNSUPPORTED, "bf16 scores support ld_te, ld_tr < 4194304");
    if (!bf16 && Q > 65535) return fail(LOGRA_ERR_UNSUPPORTED, "fp32 / fp64 scores support Q <= 65535");
    if (Q == 0) return ok();
    if (topk > 0) {
        TRY(check_dev(topk_val, "topk_val", 4));
        TRY(check_dev(topk_idx, "topk_idx", 8));
    }
    if (N_chunk == 0) {
        if (topk > 0 && !merge) {   // no candidates: every slot is padding
            const hipError_t e = logra::launch_topk(nullptr, 0, Q, 0, train_base, topk, topk_val, topk_idx,
                                                    false, static_cast<hipStream_t>(stream));
            if (e != hipSuccess) return hip_fail(e, "top-k launch");
        }
        return ok();
    }
    TRY(check_dev(g_test_pre, "g_test_pre", bf16 ? 16 : esize(te_dtype)));
    TRY(check_dev(g_train, "g_train", bf16 ? 16 : esize(tr_dtype)));
    if (row_scale) TRY(check_dev(row_scale, "row_scale", 4));
    if (col_scale) TRY(check_dev(col_scale, "col_scale", 4));
    const logra::ScoreScale scale{row_scale, col_scale};
    const size_t need = logra_influence_ws_size(Q, N_chunk, topk, scores != nullptr);
    if (need) TRY(check_ws(ws, ws_bytes, need));
    char *wp = static_cast<char *>(ws);
    float *s_buf = scores;
    int64_t ld = ld_s;
    if (scores != nullptr) {
        TRY(check_dev(scores, "scores", 4));
    } else {
        s_buf = reinterpret_cast<float *>(wp);
        ld = N_chunk;
        wp += round256(sizeof(float) * static_cast<size_t>(Q) * static_cast<size_t>(N_chunk));
    }
    const hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t pre = (bf16 && topk > 0) ? logra::topk_prefix_rows(N_chunk, topk) : 0;
    if (pre == 0) {
        hipError_t e = logra::launch_scores(g_test_pre, te_dtype, ld_te, Q, g_train, tr_dtype, ld_tr, N_chunk, D,
                                            s_buf, ld, nullptr, scale, s);
        if (e != hipSuccess) return hip_fail(e, "score launch");
        if (topk > 0) {
            e = logra::launch_topk(s_buf, ld, Q, N_chunk, train_base, topk, topk_val, topk_idx, merge != 0, s);
            if (e != hipSuccess) return hip_fail(e, "top-k launch");
        }
        return ok();
    }
    // Large chunk: exact top-k of the first `pre` rows, whose k-th values then
    // filter the scores of the rest in the GEMM epilogue; the candidates (or,
    // for a row whose candidates overflow, its full score row) are merged.
    const size_t q4 = round256(4 * static_cast<size_t>(Q));
    float *thr = reinterpret_cast<float *>(wp);
    int *cnt = reinterpret_cast<int *>(wp + q4);
    float *cval = reinterpret_cast<float *>(wp + 2 * q4);
    int *cidx = reinterpret_cast<int *>(wp + 2 * q4 + round256(4 * static_cast<size_t>(Q) * logra::kCandCap));
    hipError_t e = logra::launch_scores(g_test_pre, LOGRA_BF16, ld_te, Q, g_train, LOGRA_BF16, ld_tr, pre, D, s_buf,
                                        ld, nullptr, scale, s);
    if (e != hipSuccess) return hip_fail(e, "score launch");
    e = logra::launch_topk(s_buf, ld, Q, pre, train_base, topk, topk_val, topk_idx, merge != 0, s);
    if (e != hipSuccess) return hip_fail(e, "top-k launch");
    e = logra::launch_topk_threshold(topk_val, topk_idx, Q, topk, thr, cnt, s);
    if (e != hipSuccess) return hip_fail(e, "top-k threshold launch");
    const logra::ScoreFilter filt{thr, cnt, cval, cidx, logra::kCandCap};
    const void *tr_rest = static_cast<const uint16_t *>(g_train) + pre * ld_tr;
    const logra::ScoreScale scale_rest{row_scale, col_scale ? col_scale + pre : nullptr};
    e = logra::launch_scores(g_test_pre, LOGRA_BF16, ld_te, Q, tr_rest, LOGRA_BF16, ld_tr, N_chunk - pre, D,
                             s_buf + pre, ld, &filt, scale_rest, s);
    if (e != hipSuccess) return hip_fail(e, "score launch");
    e = logra::launch_topk_filtered(s_buf + pre, ld, Q, N_chunk - pre, train_base + pre, topk, topk_val, topk_idx,
                                    cnt, cval, cidx, logra::kCandCap, s);
    if (e != hipSuccess) return hip_fail(e, "top-k merge launch");
    return ok();
}


int logra_influence_scores(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q,
                           const void *g_train, int tr_dtype, int64_t ld_tr, int64_t N_chunk, int D,
                           int64_t train_base, float *scores, int64_t ld_s, int topk, float *topk_val,
                           int64_t *topk_idx, int merge, void *ws, size_t ws_bytes, void *stream) {
    return influence_impl(g_test_pre, te_dtype, ld_te, Q, g_train, tr_dtype, ld_tr, N_chunk, D, train_base,
                          scores, ld_s, topk, topk_val, topk_idx, merge, nullptr, nullptr, ws, ws_bytes, stream);
}

int logra_influence_scores_scaled(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q,
                                  const void *g_train, int tr_dtype, int64_t ld_tr, int64_t N_chunk, int D,
                                  int64_t train_base, const float *row_scale, const float *col_scale,
                                  float *scores, int64_t ld_s, int topk, float *topk_val, int64_t *topk_idx,
                                  int merge, void *ws, size_t ws_bytes, void *stream) {
    return influence_impl(g_test_pre, te_dtype, ld_te, Q, g_train, tr_dtype, ld_tr, N_chunk, D, train_base,
                          scores, ld_s, topk, topk_val, topk_idx, merge, row_scale, col_scale, ws, ws_bytes,
                          stream);
}

size_t logra_self_influence_ws_size(int D, int n_blocks) {
    if (D <= 0 || n_blocks <= 0) return 0;
    return round256(logra::self_influence_ws_bytes(D, n_blocks));
}

int logra_self_influence_blocks(const float *S, int D, int n_blocks, int64_t N, double damp_ratio,
                                const void *g, int g_dtype, int64_t ld, int64_t rows, float *self_out,
                                float *rsqrt_out, void *ws, size_t ws_bytes, void *stream) {
    if (!valid_dtype(g_dtype)) return fail(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if (D <= 0 || n_blocks <= 0 || rows < 0) return fail(LOGRA_ERR_INVALID_ARG, "need D > 0, n_blocks > 0, rows >= 0");
    if (D > LOGRA_MAX_PRECOND_D) return fail(LOGRA_ERR_UNSUPPORTED, "D must be <= %d", LOGRA_MAX_PRECOND_D);
    if (n_blocks > 65535) return fail(LOGRA_ERR_UNSUPPORTED, "n_blocks must be <= 65535");
    if (ld < static_cast<int64_t>(D) * n_blocks) return fail(LOGRA_ERR_INVALID_ARG, "ld must be >= D * n_blocks");
    if (damp_ratio != damp_ratio) return fail(LOGRA_ERR_INVALID_ARG, "damp_ratio is NaN");
    if (damp_ratio >= 0.0 && N <= 0) return fail(LOGRA_ERR_INVALID_ARG, "N must be > 0");
    if (rows == 0) return ok();   // nothing to factor for
    if (self_out == nullptr && rsqrt_out == nullptr)
        return fail(LOGRA_ERR_INVALID_ARG, "nothing to compute: self_out and rsqrt_out are NULL");
    const bool bf16 = g_dtype == LOGRA_BF16;
    if (bf16 && (D % 8 || ld % 8)) return fail(LOGRA_ERR_INVALID_ARG, "bf16 gradients need D and ld multiples of 8");
    if (bf16 && ld >= (int64_t{1} << 22)) return fail(LOGRA_ERR_UNSUPPORTED, "bf16 gradients support ld < 4194304");
    if ((!bf16 || D % 32) && rows > INT32_MAX)
        return fail(LOGRA_ERR_UNSUPPORTED, "fp32 gradients, or D not a multiple of 32, support rows < 2^31");
    if (damp_ratio >= 0.0) TRY(check_dev(S, "S", 4));
    if (self_out) TRY(check_dev(self_out, "self_out", 4));
    if (rsqrt_out) TRY(check_dev(rsqrt_out, "rsqrt_out", 4));
    TRY(check_ws(ws, ws_bytes, logra_self_influence_ws_size(D, n_blocks)));
    TRY(check_dev(g, "g", bf16 ? 16 : 4));
    const hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = logra::launch_inverse_factor(S, D, n_blocks, N, damp_ratio,
                                                 logra::self_influence_interleaved(bf16, D), ws, s);
    if (e != hipSuccess) return hip_fail(e, "factor launch");
    e = logra::launch_self_influence(g, bf16, ld, rows, D, n_blocks, ws, self_out, rsqrt_out, s);
    if (e != hipSuccess) return hip_fail(e, "self-influence launch");
    // synchronous, like the preconditioner, so that a non-positive pivot is reported
    return report_not_pd(ws, D, n_blocks, s);
}

// ---------------------------------------------------------------------------
// Out-of-core scoring: the store in pinned host memory, streamed in chunks.
size_t logra_influence_stream_ws_size(int Q, int64_t chunk_rows, int D, int tr_dtype, int topk) {
    if (Q < 0 || chunk_rows <= 0 || D <= 0 || !valid_dtype64(tr_dtype) || topk <= 0) return 0;
    const size_t stage = round256(static_cast<size_t>(chunk_rows) * D * esize(tr_dtype));
    return 2 * stage + logra_influence_ws_size(Q, chunk_rows, topk, 0);
}

int logra_influence_stream(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q, const void *g_train_host,
                           int tr_dtype, int64_t ld_tr, int64_t N, int D, int64_t chunk_rows, int topk,
                           float *topk_val, int64_t *topk_idx, void *ws, size_t ws_bytes, void *stream,
                           void *copy_stream) {
    TRY(check_score_dtypes(te_dtype, tr_dtype));
    if (Q < 0 || N < 0 || D <= 0 || chunk_rows <= 0)
        return fail(LOGRA_ERR_INVALID_ARG, "need Q >= 0, N >= 0, D > 0, chunk_rows > 0");
    if (topk <= 0) return fail(LOGRA_ERR_INVALID_ARG, "topk must be > 0");
    if (topk > LOGRA_MAX_TOPK) return fail(LOGRA_ERR_UNSUPPORTED, "topk must be <= %d", LOGRA_MAX_TOPK);
    if (ld_tr < D) return fail(LOGRA_ERR_INVALID_ARG, "ld_tr must be >= D");
    if (chunk_rows > INT32_MAX) return fail(LOGRA_ERR_UNSUPPORTED, "chunk_rows must be < 2^31");
    if (tr_dtype == LOGRA_BF16 && (D % 8 || ld_te % 8))
        return fail(LOGRA_ERR_INVALID_ARG, "bf16 scores need D and ld_te multiples of 8");
    if (Q == 0) return ok();
    const size_t es = esize(tr_dtype);
    if (N > 0) TRY(check_pinned(g_train_host, "g_train_host", es == 2 ? 16 : es));
    TRY(check_dev(topk_val, "topk_val", 4));
    TRY(check_dev(topk_idx, "topk_idx", 8));
    const size_t need = logra_influence_stream_ws_size(Q, chunk_rows, D, tr_dtype, topk);
    TRY(check_ws(ws, ws_bytes, need));
    const hipStream_t cs = static_cast<hipStream_t>(stream);
    const size_t stage = round256(static_cast<size_t>(chunk_rows) * D * es);
    char *buf[2] = {static_cast<char *>(ws), static_cast<char *>(ws) + stage};
    void *iws = static_cast<char *>(ws) + 2 * stage;
    const size_t iws_bytes = ws_bytes - 2 * stage;
    if (N == 0)   // an empty store: the top-k padding only
        return logra_influence_scores(g_test_pre, te_dtype, ld_te, Q, buf[0], tr_dtype, D, 0, D, 0, nullptr, 1,
                                      topk, topk_val, topk_idx, 0, iws, iws_bytes, stream);

    // Copy stream (created for the call unless given) and the events that
    // order the double buffer: chunk c fills buffer c % 2 once the scoring of
    // chunk c - 2 has released it; scoring waits for the fill.
    hipStream_t xs = static_cast<hipStream_t>(copy_stream);
    const bool own = xs == nullptr;
    hipError_t e = hipSuccess;
    if (own && (e = hipStreamCreateWithFlags(&xs, hipStreamNonBlocking)) != hipSuccess)
        return hip_fail(e, "copy stream");
    hipEvent_t filled[2] = {nullptr, nullptr}, freed[2] = {nullptr, nullptr};
    int rc = LOGRA_OK;
    for (int b = 0; b < 2 && e == hipSuccess; ++b) {
        e = hipEventCreateWithFlags(&filled[b], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&freed[b], hipEventDisableTiming);
    }
    if (e != hipSuccess) rc = hip_fail(e, "event");
    const int64_t chunks = (N + chunk_rows - 1) / chunk_rows;
    for (int64_t c = 0; c < chunks && rc == LOGRA_OK; ++c) {
        const int b = static_cast<int>(c & 1);
        const int64_t r0 = c * chunk_rows, rows = N - r0 < chunk_rows ? N - r0 : chunk_rows;
        const char *src = static_cast<const char *>(g_train_host) + static_cast<size_t>(r0) * ld_tr * es;
        if (c >= 2 && (e = hipStreamWaitEvent(xs, freed[b], 0)) != hipSuccess) {
            rc = hip_fail(e, "wait for a free buffer");
            break;
        }
        e = ld_tr == D ? hipMemcpyAsync(buf[b], src, static_cast<size_t>(rows) * D * es, hipMemcpyHostToDevice, xs)
                       : hipMemcpy2DAsync(buf[b], D * es, src, ld_tr * es, D * es, static_cast<size_t>(rows),
                                          hipMemcpyHostToDevice, xs);
        if (e == hipSuccess) e = hipEventRecord(filled[b], xs);
        if (e == hipSuccess) e = hipStreamWaitEvent(cs, filled[b], 0);
        if (e != hipSuccess) {
            rc = hip_fail(e, "chunk copy");
            break;
        }
        rc = logra_influence_scores(g_test_pre, te_dtype, ld_te, Q, buf[b], tr_dtype, D, rows, D, r0, nullptr, 1,
                                    topk, topk_val, topk_idx, c > 0, iws, iws_bytes, stream);
        if (rc == LOGRA_OK && (e = hipEventRecord(freed[b], cs)) != hipSuccess) rc = hip_fail(e, "event record");
    }
    // synchronous: the buffers, events and (own) stream live until the last chunk is scored
    e = hipStreamSynchronize(cs);
    if (rc == LOGRA_OK && e != hipSuccess) rc = hip_fail(e, "stream synchronize");
    e = hipStreamSynchronize(xs);
    if (rc == LOGRA_OK && e != hipSuccess) rc = hip_fail(e, "copy stream synchronize");
    for (int b = 0; b < 2; ++b) {
        if (filled[b]) (void)hipEventDestroy(filled[b]);
        if (freed[b]) (void)hipEventDestroy(freed[b]);
    }
    if (own) (void)hipStreamDestroy(xs);
    return rc == LOGRA_OK ? ok() : rc;
}

int logra_offload_rows(const void *src, int64_t ld_src, void *dst, int64_t ld_dst, int64_t rows, int64_t row_bytes,
                       void *stream, void *copy_stream, void *done) {
    if (rows < 0 || row_bytes <= 0) return fail(LOGRA_ERR_INVALID_ARG, "need rows >= 0 and row_bytes > 0");
    if (ld_src < row_bytes || ld_dst < row_bytes)
        return fail(LOGRA_ERR_INVALID_ARG, "row strides must be >= row_bytes");
    if (rows == 0) return ok();
    const int64_t last_src = (rows - 1) * ld_src + row_bytes - 1, last_dst = (rows - 1) * ld_dst + row_bytes - 1;
    TRY(check_dev(src, "src", 1));
    TRY(check_dev(static_cast<const char *>(src) + last_src, "the last row of src", 1));
    TRY(check_pinned(dst, "dst", 1));
    TRY(check_pinned(static_cast<char *>(dst) + last_dst, "the last row of dst", 1));
    const hipStream_t cs = static_cast<hipStream_t>(stream);
    hipStream_t xs = copy_stream ? static_cast<hipStream_t>(copy_stream) : cs;
    hipError_t e = hipSuccess;
    if (xs != cs) {
        // the copy waits for the work enqueued on `stream` so far.  One event
        // per thread and device serves every call: a wait takes the event's
        // state when it is enqueued, so re-recording it later is harmless,
        // and no call destroys an event that may still be pending.
        int dev = 0;
        if ((e = hipGetDevice(&dev)) != hipSuccess) return hip_fail(e, "current device");
        static thread_local hipEvent_t ready[64] = {};
        if (dev < 0 || dev >= 64) return fail(LOGRA_ERR_UNSUPPORTED, "device index %d >= 64", dev);
        if (!ready[dev] && (e = hipEventCreateWithFlags(&ready[dev], hipEventDisableTiming)) != hipSuccess)
            return hip_fail(e, "event");
        e = hipEventRecord(ready[dev], cs);
        if (e == hipSuccess) e = hipStreamWaitEvent(xs, ready[dev], 0);
        if (e != hipSuccess) return hip_fail(e, "order the copy after the stream");
    }
    e = ld_src == row_bytes && ld_dst == row_bytes
            ? hipMemcpyAsync(dst, src, static_cast<size_t>(rows * row_bytes), hipMemcpyDeviceToHost, xs)
            : hipMemcpy2DAsync(dst, static_cast<size_t>(ld_dst), src, static_cast<size_t>(ld_src),
                               static_cast<size_t>(row_bytes), static_cast<size_t>(rows), hipMemcpyDeviceToHost, xs);
    if (e != hipSuccess) return hip_fail(e, "device-to-host copy");
    if (done && (e = hipEventRecord(static_cast<hipEvent_t>(done), xs)) != hipSuccess)
        return hip_fail(e, "record done");
    return ok();
}

size_t logra_act_cov_ws_size(int B, int T) {
    if (B <= 0 || T <= 0) return 0;
    return round256(logra::act_cov_ws_bytes(B, T));
}

int logra_act_cov_accumulate(const void *a, int a_dtype, int B, int T, int n, const uint8_t *mask, float *C,
                             void *ws, size_t ws_bytes, void *stream) {
    if (!valid_dtype(a_dtype)) return fail(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if (B < 0 || T < 0 || n <= 0) return fail(LOGRA_ERR_INVALID_ARG, "need B >= 0, T >= 0, n > 0");
    const bool bf16 = a_dtype == LOGRA_BF16;
    if (bf16 && n % 8) return fail(LOGRA_ERR_INVALID_ARG, "bf16 activations need n a multiple of 8");
    if (n > (1 << 20)) return fail(LOGRA_ERR_UNSUPPORTED, "n must be <= 1048576");
    if (static_cast<int64_t>(B) * T > INT32_MAX) return fail(LOGRA_ERR_UNSUPPORTED, "B * T must be < 2^31");
    if (B == 0 || T == 0) return ok();
    TRY(check_dev(a, "a", bf16 ? 16 : 4));
    TRY(check_dev(C, "C", 4));
    if (mask) TRY(check_dev(mask, "mask", 1));
    TRY(check_ws(ws, ws_bytes, logra_act_cov_ws_size(B, T)));
    hipError_t e = logra::launch_act_cov(a, bf16, B, T, n, mask, C, ws, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "activation covariance launch");
    return ok();
}

int logra_act_cov_accumulate_group(const logra_act_cov_desc *factors, int n_desc, int a_dtype, int B, int T,
                                   const uint8_t *mask, void *ws, size_t ws_bytes, void *stream) {
    static_assert(LOGRA_MAX_ACT_COV_GROUP == logra::kMaxActCovGroup, "one group limit");
    if (factors == nullptr) return fail(LOGRA_ERR_INVALID_ARG, "factors is NULL");
    if (n_desc < 1 || n_desc > LOGRA_MAX_ACT_COV_GROUP)
        return fail(n_desc > LOGRA_MAX_ACT_COV_GROUP ? LOGRA_ERR_UNSUPPORTED : LOGRA_ERR_INVALID_ARG,
                    "n_desc must be in 1..%d", LOGRA_MAX_ACT_COV_GROUP);
    if (!valid_dtype(a_dtype)) return fail(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if (B < 0 || T < 0) return fail(LOGRA_ERR_INVALID_ARG, "need B >= 0, T >= 0");
    const bool bf16 = a_dtype == LOGRA_BF16;
    for (int f = 0; f < n_desc; ++f) {
        const int n = factors[f].n;
        if (n <= 0) return fail(LOGRA_ERR_INVALID_ARG, "factor %d: need n > 0", f);
        if (bf16 && n % 8) return fail(LOGRA_ERR_INVALID_ARG, "factor %d: bf16 activations need n a multiple of 8", f);
        if (n > (1 << 20)) return fail(LOGRA_ERR_UNSUPPORTED, "factor %d: n must be <= 1048576", f);
    }
    if (static_cast<int64_t>(B) * T > INT32_MAX) return fail(LOGRA_ERR_UNSUPPORTED, "B * T must be < 2^31");
    if (B == 0 || T == 0) return ok();
    const void *a[LOGRA_MAX_ACT_COV_GROUP];
    float *C[LOGRA_MAX_ACT_COV_GROUP];
    int n[LOGRA_MAX_ACT_COV_GROUP];
    for (int f = 0; f < n_desc; ++f) {
        a[f] = factors[f].a;
        C[f] = factors[f].C;
        n[f] = factors[f].n;
    }
    // tiles of different factors run at the same time: two C that share bytes would race
    for (int f = 0; f < n_desc; ++f)
        for (int h = 0; h < f; ++h) {
            const uintptr_t f0 = reinterpret_cast<uintptr_t>(C[f]), h0 = reinterpret_cast<uintptr_t>(C[h]);
            const uintptr_t f1 = f0 + static_cast<uintptr_t>(n[f]) * n[f] * sizeof(float);
            const uintptr_t h1 = h0 + static_cast<uintptr_t>(n[h]) * n[h] * sizeof(float);
            if (f0 < h1 && h0 < f1) return fail(LOGRA_ERR_INVALID_ARG, "C of factors %d and %d overlap", h, f);
        }
    for (int f = 0; f < n_desc; ++f) {
        TRY(check_dev(a[f], "a", bf16 ? 16 : 4));
        TRY(check_dev(C[f], "C", 4));
    }
    if (mask) TRY(check_dev(mask, "mask", 1));
    TRY(check_ws(ws, ws_bytes, logra_act_cov_ws_size(B, T)));
    hipError_t e = logra::launch_act_cov_group(a, C, n, n_desc, bf16, B, T, mask, ws, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "activation covariance launch");
    return ok();
}

size_t logra_pca_ws_size(int n, int k) {
    if (n <= 0 || k <= 0 || k > n || k > LOGRA_MAX_PCA_K) return 0;
    return round256(logra::pca_ws_bytes(n, k));
}

int logra_pca_topk(const float *C, int n, int k, int iters, void *P, int P_dtype, int64_t ld_p, float *eigvals,
                   void *ws, size_t ws_bytes, void *stream) {
    if (!valid_dtype(P_dtype)) return fail(LOGRA_ERR_INVALID_ARG, "bad dtype");
    if (n <= 0 || k <= 0 || k > n) return fail(LOGRA_ERR_INVALID_ARG, "need 1 <= k <= n");
    if (k > LOGRA_MAX_PCA_K) return fail(LOGRA_ERR_UNSUPPORTED, "k must be <= %d", LOGRA_MAX_PCA_K);
    if (n > 65536) return fail(LOGRA_ERR_UNSUPPORTED, "n must be <= 65536");
    if (iters < 1 || iters > 100000) return fail(LOGRA_ERR_INVALID_ARG, "need 1 <= iters <= 100000");
    if (ld_p < n) return fail(LOGRA_ERR_INVALID_ARG, "ld_p must be >= n");
    TRY(check_dev(C, "C", 4));
    TRY(check_dev(P, "P", P_dtype == LOGRA_BF16 ? 2 : 4));
    if (eigvals) TRY(check_dev(eigvals, "eigvals", 4));
    TRY(check_ws(ws, ws_bytes, logra_pca_ws_size(n, k)));
    hipError_t e = logra::launch_pca_topk(C, n, k, iters, P, P_dtype == LOGRA_BF16, ld_p, eigvals, ws,
                                          static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "pca launch");
    return ok();
}

}  // extern "C"
