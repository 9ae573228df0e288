// Host-side launch interface between the C ABI and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "logra.h"

namespace logra {

// Host-side entry used by both projection entry points (abi.cpp): argument
// checks, then the launches; ws_known skips the pointer check of a workspace
// that the library itself owns.
int project_layers_checked(const logra_layer_desc *layers, int n_layers, int in_dtype, int B, int T,
                           const uint8_t *mask, int k_in, int k_out, int g_dtype, int64_t g_ld, void *ws,
                           size_t ws_bytes, bool ws_known, void *stream);
// Sets the thread's error message; returns LOGRA_ERR_HIP / LOGRA_ERR_UNSUPPORTED.
int hip_fail(hipError_t e, const char *what);
int fail_unsupported(const char *msg);
int fail_code(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));   // sets the message
int ok_code();                                                                         // clears it
int check_pinned_code(const void *p, const char *name, size_t align);                  // pinned host memory

typedef uint16_t bf16_bits_t;   // a bf16 value as its bit pattern
enum DtypeCode { kF32 = 0, kBF16 = 1, kF64 = 2 };   // element types, numbered as in the C ABI
constexpr int kMaxGroup = 48;   // layers per grouped projection launch
constexpr int kMaxK = 128;
constexpr int kMaxTopk = 1024;
constexpr int kMaxPrecondD = 8192;

// Workspace regions are carved at 256-byte boundaries.
__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

struct ProjLayer {
    const void *x;
    const void *dy;
    const void *p_in;
    const void *p_out;
    void *g_out;
    int n_in;
    int n_out;
};

struct ProjGroup {
    ProjLayer layer[kMaxGroup];
    int n_layers;
};

// Projection (Sec. 3.1 Eq. (5)): chunk partials and per-tile sums in the
// workspace, then a fixed-order sum over tiles into each layer's g_out rows.
size_t project_ws_bytes(const int *n_in, const int *n_out, int n_layers, int B, int T, int k_in,
                        int k_out);
hipError_t launch_project(const ProjGroup &grp, bool bf16_in, int B, int T, const uint8_t *mask,
                          int k_in, int k_out, bool bf16_out, int64_t g_ld, void *ws, hipStream_t s);

// Covariance S_l += G_l^T G_l for n_blocks column blocks of width D; the
// _f64 form keeps S in float64 (rows fp32, or fp64 when f64_rows).
hipError_t launch_cov(const void *g, bool bf16, int64_t ld, int B, int D, int n_blocks, float *S, bool lower,
                      hipStream_t s);
hipError_t launch_cov_f64(const void *g, bool f64_rows, int64_t ld, int B, int D, int n_blocks, double *S,
                          hipStream_t s);

// Damped Cholesky preconditioning of n_blocks blocks.  Writes a per-block
// status word into the workspace; precond_info_ptr() locates it.
size_t precond_ws_bytes(int D, int n_blocks, int Q);
int *precond_info_ptr(void *ws, int D, int n_blocks);
// S is fp32, or fp64 when s_f64; in_dt / out_dt are DtypeCode values.
hipError_t launch_precondition(const void *S, bool s_f64, int D, int n_blocks, int64_t N, double damp_ratio,
                               const void *g_test, int in_dt, int64_t ld_in, int Q, void *g_out, int out_dt,
                               int64_t ld_out, void *ws, hipStream_t s);
hipError_t launch_copy_rows(const void *src, int in_dt, int64_t ld_in, int rows, int cols,
                            void *dst, int out_dt, int64_t ld_out, hipStream_t s);

// Self-influence (l-RelatIF's normaliser): per block, W = L^{-1} of the
// damped covariance's Cholesky factor (identity when damp_ratio < 0), kept as
// bf16 hi + lo halves in the workspace after the preconditioner's layout;
// then self_j = sum over blocks of |W_l g_jl|^2.  Rows of W are padded with
// zeros to Dp = D rounded up to 256.  Two layouts of the halves:
//  - split: hi [n_blocks][Dp][D], then lo likewise (self_influence_w);
//  - interleaved (bf16 gradients with D a multiple of 64): one array
//    [n_blocks][Dp][2D] at self_influence_w(.., false) whose row o holds,
//    for each 64-column chunk c, hi of the chunk then lo of the chunk.
inline bool self_influence_interleaved(bool bf16, int D) { return bf16 && D % 64 == 0; }
size_t self_influence_ws_bytes(int D, int n_blocks);
bf16_bits_t *self_influence_w(void *ws, int D, int n_blocks, bool lo);
hipError_t launch_inverse_factor(const float *S, int D, int n_blocks, int64_t N, double damp_ratio,
                                 bool interleaved, void *ws, hipStream_t s);
hipError_t launch_self_influence(const void *g, bool bf16, int64_t ld, int64_t rows, int D, int n_blocks,
                                 const void *ws, float *self_out, float *rsqrt_out, hipStream_t s);

// KFAC activation covariance (the PCA initialisation of P): C [n][n] fp32 +=
// sum over unmasked tokens of a_t a_t^T for a [B][T][n]; workspace holds the
// list of non-empty 32-token slabs.
size_t act_cov_ws_bytes(int B, int T);
hipError_t launch_act_cov(const void *a, bool bf16, int B, int T, int n, const uint8_t *mask, float *C, void *ws,
                          hipStream_t s);
// The same for `count` (<= kMaxActCovGroup) factors of one batch in one launch:
// a[i] [B][T][n[i]] into C[i] [n[i]][n[i]]; the factors share B, T, the mask
// and the dtype, and their C must not overlap.  Each factor's result is
// identical to launch_act_cov's.
constexpr int kMaxActCovGroup = 32;
hipError_t launch_act_cov_group(const void *const *a, float *const *C, const int *n, int count, bool bf16, int B,
                                int T, const uint8_t *mask, void *ws, hipStream_t s);

// Top-k eigenvectors of a symmetric PSD fp32 C [n][n] (k <= 64) as the rows
// of P [k][ld_p], by subspace iteration with Rayleigh-Ritz extraction.
size_t pca_ws_bytes(int n, int k);
hipError_t launch_pca_topk(const float *C, int n, int k, int iters, void *P, bool bf16_out, int64_t ld_p,
                           float *eigvals, void *ws, hipStream_t s);

// Score GEMM s = te * tr^T (fp32 result) and per-query top-k.  With a
// filter (bf16 only), scores at or above thr[q] are also appended to row q's
// candidate list: cnt[q] counts them (past `cap` too), val/idx hold the
// first `cap` of them (idx = column within this launch).
constexpr int kCandCap = 8192;   // candidates kept per query row
struct ScoreFilter {
    const float *thr;
    int *cnt;
    float *val;
    int *idx;
    int cap;
};
// Optional scales of normalised scores: s[q][j] * row[q] * col[j] (NULL = 1;
// col is indexed by the column of this launch).
struct ScoreScale {
    const float *row;
    const float *col;
};
// te_dt / tr_dt: both kBF16 (bf16 MFMA), or each kF32 or kF64 (float64
// accumulation, no filter).
hipError_t launch_scores(const void *te, int te_dt, int64_t ld_te, int Q, const void *tr, int tr_dt,
                         int64_t ld_tr, int64_t N, int D, float *s, int64_t ld_s, const ScoreFilter *filt,
                         const ScoreScale &scale, hipStream_t st);
// Rows of a chunk scored and selected exactly before candidate filtering
// starts (their running top-k sets the thresholds); 0 = no filtering.
int64_t topk_prefix_rows(int64_t N, int k);
hipError_t launch_topk(const float *s, int64_t ld_s, int Q, int64_t N, int64_t base, int k,
                       float *val, int64_t *idx, bool merge, hipStream_t st);
hipError_t launch_topk_threshold(const float *val, const int64_t *idx, int Q, int k, float *thr,
                                 int *cnt, hipStream_t st);
hipError_t launch_topk_filtered(const float *s, int64_t ld_s, int Q, int64_t N, int64_t base, int k,
                                float *val, int64_t *idx, const int *cnt, const float *cval,
                                const int *cidx, int cap, hipStream_t st);

}  // namespace logra
