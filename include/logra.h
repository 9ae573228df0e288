/*
 * logra.h -- C ABI of the LoGra hot path on AMD Instinct MI355X (gfx950).
 *
 * LoGra (Choe et al., arXiv 2405.13954) values training data with influence
 * functions computed in a low-dimensional gradient space.  This library
 * implements the data-parallel hot path of that method:
 *
 *   logging   : per-example structured gradient projection (Sec. 3.1, Eq. (5))
 *               and the projected Fisher covariance (Sec. 2 Eq. (3); App. D)
 *   influence : damped inverse applied to test gradients (Sec. 2 Eq. (2),
 *               step (1); damping of App. C), the score GEMM against stored
 *               training gradients (Eq. (2), step (2)) and per-query top-k.
 *
 * Conventions shared by every entry point
 *   - Tensors are caller-owned DEVICE memory (hipMalloc or a framework
 *     allocator).  Host pointers are rejected with LOGRA_ERR_INVALID_ARG.
 *     The library allocates no device memory; scratch space ("workspace") is
 *     passed in by the caller after a *_ws_size query.
 *   - Arrays are row-major with the last index contiguous; a "leading
 *     dimension" (ld) is a row stride in ELEMENTS.
 *   - Base pointers and row strides in bytes must be multiples of 16 (the
 *     kernels use 128-bit loads); otherwise LOGRA_ERR_INVALID_ARG.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued
 *     on it and the call returns without waiting, except where stated.
 *   - Calls return a logra_status and never abort; logra_last_error() gives a
 *     thread-local message for the last non-OK return.  Kernel faults surface
 *     as HIP errors at the caller's next synchronisation.
 *   - bf16 outputs are rounded from fp32 to nearest, ties to even.
 *   - All functions are reentrant; calls that share an output buffer must be
 *     ordered by the caller (same stream or events).
 */
#ifndef LOGRA_H
#define LOGRA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    LOGRA_OK = 0,
    LOGRA_ERR_INVALID_ARG = -1, /* bad pointer, size, stride, alignment or dtype */
    LOGRA_ERR_UNSUPPORTED = -2, /* valid request beyond a compiled limit */
    LOGRA_ERR_HIP = -3,         /* a HIP runtime call failed */
    LOGRA_ERR_NOT_PD = -4,      /* damped covariance is not positive definite */
    LOGRA_ERR_WORKSPACE = -5,   /* workspace missing or smaller than *_ws_size */
    LOGRA_ERR_IO = -6           /* a store file read or write failed or came up short */
} logra_status;

/* Element types.  LOGRA_F64 is accepted only where a call says so: the
 * float64 statistics path of fp32 workloads (covariance, preconditioned test
 * gradients and the scores against them). */
typedef enum { LOGRA_F32 = 0, LOGRA_BF16 = 1, LOGRA_F64 = 2 } logra_dtype;

/* Compiled limits. */
#define LOGRA_MAX_K 128          /* k_in, k_out of one projection */
#define LOGRA_MAX_GROUP 48       /* layers in one logra_project_layers call */
#define LOGRA_MAX_PRECOND_D 8192 /* dimension of one preconditioner block */
#define LOGRA_MAX_TOPK 1024

const char *logra_last_error(void);
const char *logra_version(void);

/* ------------------------------------------------------------------------
 * Per-example structured gradient projection of one linear layer
 * (Sec. 3.1, Eq. (4)-(5)):
 *
 *     G_b = sum_{t : mask[b,t] != 0}  (P_out dy_{b,t}) (P_in x_{b,t})^T
 *
 * the k_out x k_in projected gradient of example b, formed from the
 * projected activations without materialising the n_out x n_in gradient.
 * The sum runs over tokens (summed, not averaged, loss).
 *
 *   x      [B][T][n_in]   layer inputs (forward activations), in_dtype
 *   dy     [B][T][n_out]  gradients w.r.t. the layer outputs, in_dtype
 *   mask   [B][T] uint8   token t of example b contributes iff mask != 0;
 *                         NULL = every token contributes.  Masked tokens are
 *                         never read: their contribution is exactly zero even
 *                         if their slots hold NaN or Inf.
 *   p_in   [k_in][n_in]   and p_out [k_out][n_out], in_dtype
 *   g_out  row b of the result is written at g_out + b * g_ld (elements),
 *          flattened out-major: element o * k_in + i holds G_b[o][i].
 *          g_dtype F32 or BF16.  Rows may interleave with other layers'
 *          columns of a gradient store (g_ld >= k_in * k_out).
 *   ws     workspace of at least logra_project_ws_size(B, T, n_in, n_out,
 *          k_in, k_out) bytes (fp32 partial sums, about
 *          B * T * (n_in + n_out) / 2048 * 16 * ceil(k/16) * 4 bytes);
 *          contents on entry are ignored.
 * Limits: n_in, n_out multiples of 8 (bf16) or 4 (fp32); 1 <= k <= LOGRA_MAX_K.
 * B = 0 or T = 0 is a no-op.  Deterministic: reruns are bitwise identical.
 * ---------------------------------------------------------------------- */
size_t logra_project_ws_size(int B, int T, int n_in, int n_out, int k_in, int k_out);
int logra_project_layer(const void *x, const void *dy, int in_dtype, int B, int T, int n_in,
                        int n_out, const uint8_t *mask, const void *p_in, const void *p_out,
                        int k_in, int k_out, void *g_out, int g_dtype, int64_t g_ld, void *ws,
                        size_t ws_bytes, void *stream);

/* The same projection for up to LOGRA_MAX_GROUP layers of one batch in one
 * launch (the layers share B, T, mask, k_in, k_out, dtypes and g_ld; each has
 * its own tensors and output base).  Results are identical to calling
 * logra_project_layer once per layer. */
typedef struct {
    const void *x;
    const void *dy;
    const void *p_in;
    const void *p_out;
    void *g_out;
    int n_in;
    int n_out;
} logra_layer_desc;

size_t logra_project_layers_ws_size(const logra_layer_desc *layers, int n_layers, int B, int T,
                                    int k_in, int k_out);
int logra_project_layers(const logra_layer_desc *layers, int n_layers, int in_dtype, int B, int T,
                         const uint8_t *mask, int k_in, int k_out, int g_dtype, int64_t g_ld,
                         void *ws, size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * logra_project_layers without a workspace argument.  The workspace is a
 * static device array of the library, LOGRA_NOALLOC_WS_BYTES (64 MiB) on each
 * GPU it runs on, held until the process ends; the call allocates nothing.
 * Results are bitwise those of logra_project_layers.  A batch whose
 * logra_project_layers_ws_size exceeds LOGRA_NOALLOC_WS_BYTES returns
 * LOGRA_ERR_UNSUPPORTED (e.g. 7 Llama3-8B layers at k = 16 with B = 8,
 * T = 2048 need 16 MiB, 28 of them 63 MiB; at k = 64 with B = 16, T = 1024
 * the 7 layers need 84 MiB).
 * Calls that overlap on one GPU (other streams or threads) share the array
 * and race: order them.  Other errors as logra_project_layers. */
#define LOGRA_NOALLOC_WS_BYTES (64u * 1024u * 1024u)
int logra_project_layers_noalloc(const logra_layer_desc *layers, int n_layers, int in_dtype, int B, int T,
                                 const uint8_t *mask, int k_in, int k_out, int g_dtype, int64_t g_ld,
                                 void *stream);

/* ------------------------------------------------------------------------
 * Projected Fisher covariance (Sec. 2 Eq. (3) P H P^T; App. D Assumption 1:
 * the empirical Fisher over training examples):
 *
 *     S += sum_{b < B} g_b g_b^T
 *
 *   g   B rows of D elements at row stride ld (elements), g_dtype F32/BF16
 *   S   [D][D] fp32, caller-initialised (zero for a new statistic), updated
 *       in place and kept exactly symmetric (the upper triangle is computed
 *       and mirrored).  The caller tracks the example count N; S is not
 *       normalised here.
 * bf16 inputs use bf16 MFMA with fp32 accumulation; fp32 inputs use fp32
 * arithmetic.  B = 0 is a no-op.  Deterministic.
 * ---------------------------------------------------------------------- */
int logra_cov_accumulate(const void *g, int g_dtype, int64_t ld, int B, int D, float *S,
                         void *stream);

/* Block-diagonal form for many layers at once: columns [l*D, (l+1)*D) of g
 * update S + l*D*D, for l < n_blocks.  Same semantics per block. */
int logra_cov_accumulate_blocks(const void *g, int g_dtype, int64_t ld, int B, int D,
                                int n_blocks, float *S, void *stream);

/* The same update applied to the lower triangle alone (the symmetric rank-B
 * update of a packed-by-convention symmetric matrix, as BLAS SYRK with
 * uplo = lower): entries S[i][j] with i >= j of each block are read and
 * written; entries above the diagonal are neither read nor written.  The
 * preconditioning and inverse-factor entry points below read only the lower
 * triangle and the diagonal, so a statistic kept this way feeds them
 * directly, for two thirds of the memory traffic of the symmetric form.
 * Arguments and errors as logra_cov_accumulate_blocks. */
int logra_cov_accumulate_blocks_lower(const void *g, int g_dtype, int64_t ld, int B, int D,
                                      int n_blocks, float *S, void *stream);

/* The same statistic kept in float64, for fp32 workloads whose downstream
 * solve is ill-conditioned (the damped inverse of App. C amplifies the
 * rounding of an fp32 S by up to the condition number of C + lambda I):
 *   g   B rows of n_blocks * D elements at stride ld, g_dtype F32 or F64
 *   S   [n_blocks][D][D] fp64, caller-initialised, updated in place, kept
 *       exactly symmetric.
 * Every product and sum is formed in float64 (a product of two fp32 values
 * is exact there).  Errors as logra_cov_accumulate_blocks; a bf16 g is
 * INVALID_ARG. */
int logra_cov_accumulate_f64(const void *g, int g_dtype, int64_t ld, int B, int D, int n_blocks,
                             double *S, void *stream);

/* ------------------------------------------------------------------------
 * Damped inverse applied to test gradients, for one layer block (the iHVP
 * step (1) of Sec. 2 Eq. (2) in the projected space of Eq. (3)):
 *
 *     C = S / N,   lambda = damp_ratio * tr(C) / D   (damp_ratio x the mean
 *                                                     eigenvalue, App. C)
 *     g_out[q] = (C + lambda I)^{-1} g_test[q]        for q < Q
 *
 * computed by a float64 Cholesky factorisation and two triangular solves.
 * damp_ratio < 0 selects the identity preconditioner (g_out = g_test).
 *
 *   S       [D][D] fp32 covariance from logra_cov_accumulate or
 *           logra_cov_accumulate_blocks_lower (only the lower triangle and the
 *           diagonal are read); N > 0 the number of examples accumulated into it
 *   g_test  Q rows of D at stride ld_in, in_dtype;  g_out Q rows of D at
 *           stride ld_out, out_dtype (may not alias g_test); each of F32,
 *           BF16 or F64
 *   ws      workspace of logra_precondition_ws_size(D, 1, Q) bytes
 * SYNCHRONOUS: waits for `stream`, so that a non-positive pivot can be
 * returned as LOGRA_ERR_NOT_PD (g_out is then unspecified).
 * D <= LOGRA_MAX_PRECOND_D.
 * ---------------------------------------------------------------------- */
size_t logra_precondition_ws_size(int D, int n_blocks, int Q);
int logra_precondition(const float *S, int D, int64_t N, double damp_ratio, const void *g_test,
                       int in_dtype, int64_t ld_in, int Q, void *g_out, int out_dtype,
                       int64_t ld_out, void *ws, size_t ws_bytes, void *stream);

/* Block-diagonal form: block l uses S + l*D*D and columns [l*D, (l+1)*D) of
 * g_test and g_out, each with its own lambda_l.  NOT_PD if any block fails
 * (logra_last_error names the first). */
int logra_precondition_blocks(const float *S, int D, int n_blocks, int64_t N, double damp_ratio,
                              const void *g_test, int in_dtype, int64_t ld_in, int Q, void *g_out,
                              int out_dtype, int64_t ld_out, void *ws, size_t ws_bytes,
                              void *stream);

/* logra_precondition_blocks with S in float64 (from logra_cov_accumulate_f64);
 * same workspace size, semantics and errors.  With fp64 g_out the float64
 * solution is stored unrounded. */
int logra_precondition_f64(const double *S, int D, int n_blocks, int64_t N, double damp_ratio,
                           const void *g_test, int in_dtype, int64_t ld_in, int Q, void *g_out,
                           int out_dtype, int64_t ld_out, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Influence scores and per-query top-k (Sec. 2 Eq. (2) step (2): the dot
 * product of each preconditioned test gradient with every stored training
 * gradient; with a block-diagonal Hessian this is one dot product over the
 * concatenated layer blocks; top-k of the most valuable data, Sec. 4.1):
 *
 *     s[q][j] = sum_{d < D} g_test_pre[q][d] * g_train[j][d]
 *
 *   g_test_pre  Q rows at stride ld_te;  g_train N_chunk rows at stride ld_tr.
 *               Both BF16 (bf16 MFMA, fp32 accumulation), or each F32 or
 *               F64: then every product and sum is formed in float64 and the
 *               score rounded once to fp32 (the path of fp32 workloads, whose
 *               scores can cancel by orders of magnitude).  A bf16 operand
 *               with a non-bf16 one is UNSUPPORTED.
 *   scores      optional [Q][ld_s] fp32 output (NULL = not materialised by
 *               the caller; it then lives in the workspace).
 *   topk        0 = no selection; else 1..LOGRA_MAX_TOPK entries per query
 *               into topk_val [Q][topk] (fp32) and topk_idx [Q][topk]
 *               (int64 global train index train_base + j), sorted by value
 *               descending, ties to the lower index.  Slots beyond the
 *               number of candidates hold (-inf, -1).
 *   merge       0: the top-k buffers are overwritten with this chunk's top-k;
 *               1: they hold a running top-k (from earlier chunks) that is
 *               merged with this chunk's candidates.  Calling once per chunk
 *               with merge=1 after the first gives the top-k of all chunks.
 *   ws          workspace of logra_influence_ws_size(Q, N_chunk, topk,
 *               scores != NULL) bytes (0 when scores are given and topk = 0):
 *               the scores when not given, and for long bf16 chunks the
 *               per-query top-k candidate lists described below.
 * Long bf16 chunks (N_chunk at least twice a prefix of max(4096, about
 * 2 * topk * N_chunk / 8192) rows) select in two stages: the exact top-k of
 * the prefix gives each query a threshold (its k-th value, a lower bound on
 * the chunk's k-th value), the GEMM keeps the later scores at or above it as
 * candidates (up to 8192 per query), and the candidates are merged; a query
 * whose candidates overflow is selected from its full score row.  The result
 * is the same exact top-k in every case.
 * N_chunk < 2^31; for bf16, ld_te and ld_tr < 2^22.
 * Scores of NaN order unspecified.
 * ---------------------------------------------------------------------- */
size_t logra_influence_ws_size(int Q, int64_t N_chunk, int topk, int scores_given);
int logra_influence_scores(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q,
                           const void *g_train, int tr_dtype, int64_t ld_tr, int64_t N_chunk,
                           int D, int64_t train_base, float *scores, int64_t ld_s, int topk,
                           float *topk_val, int64_t *topk_idx, int merge, void *ws,
                           size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Normalised influence scores (l-RelatIF, Sec. 4.2: each score divided by the
 * training example's self-influence, which penalises outliers with large
 * gradient norms; the cosine form also divides by the test example's):
 *
 *     self_j   = sum_l g_jl^T (C_l + lambda_l I)^{-1} g_jl     (blocks l)
 *     s'[q][j] = s[q][j] * row_scale[q] * col_scale[j]
 *
 * with row_scale = 1/sqrt(self_test) (cosine) or 1 (l-RelatIF) and
 * col_scale = 1/sqrt(self_train).
 *
 * logra_self_influence_blocks: for `rows` gradients g (rows at stride ld,
 * n_blocks column blocks of width D, g_dtype F32 or BF16) writes self_out[j]
 * and/or rsqrt_out[j] = 1/sqrt(self_j) (0 where self_j <= 0), fp32 device
 * arrays of `rows` (either may be NULL, not both; rows = 0 returns at once).  C_l, lambda_l are formed
 * from S + l*D*D and N with damp_ratio as in logra_precondition_blocks
 * (damp_ratio < 0: identity, self_j = |g_j|^2).  The inverse Cholesky factor
 * of each block is formed in float64 and applied as two bf16 halves (about 16
 * significant bits) on the matrix cores with fp32 accumulation.
 *   ws  workspace of logra_self_influence_ws_size(D, n_blocks) bytes.
 * SYNCHRONOUS (returns LOGRA_ERR_NOT_PD like the preconditioner).
 * D <= LOGRA_MAX_PRECOND_D; bf16: D, ld multiples of 8, ld < 2^22.
 *
 * logra_influence_scores_scaled: logra_influence_scores with the scales
 * applied to every score before it is stored and before the top-k (row_scale
 * [Q], col_scale [N_chunk] indexed like the chunk's rows; NULL = 1), so the
 * top-k is the top-k of the normalised scores.
 * ---------------------------------------------------------------------- */
size_t logra_self_influence_ws_size(int D, int n_blocks);
int logra_self_influence_blocks(const float *S, int D, int n_blocks, int64_t N, double damp_ratio,
                                const void *g, int g_dtype, int64_t ld, int64_t rows, float *self_out,
                                float *rsqrt_out, void *ws, size_t ws_bytes, void *stream);
int logra_influence_scores_scaled(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q,
                                  const void *g_train, int tr_dtype, int64_t ld_tr, int64_t N_chunk, int D,
                                  int64_t train_base, const float *row_scale, const float *col_scale,
                                  float *scores, int64_t ld_s, int topk, float *topk_val, int64_t *topk_idx,
                                  int merge, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Out-of-core scoring.  The store of projected training gradients outgrows
 * GPU memory at scale (Table 1: 3.5 TB for Llama3-8B on 1B tokens), and the
 * paper hides the data IO by overlapping the reading of training gradients
 * with the influence computation (Sec. 4.2, Efficiency).
 *
 * logra_influence_stream: the running top-k of logra_influence_scores over a
 * store in PINNED HOST memory (hipHostMalloc; pageable memory is rejected),
 * g_train_host [N][ld_tr] of tr_dtype, streamed over PCIe in chunks of
 * chunk_rows rows: chunk c is copied into device staging buffer c % 2 on a
 * copy stream while chunk c - 1 is scored on `stream` (events order the
 * reuse of the two buffers).  topk_val / topk_idx [Q][topk] (device) get the
 * top-k over all N rows with global indices 0..N-1, exactly as one
 * logra_influence_scores call over the whole store would give them (N = 0:
 * padding).  copy_stream: a hipStream_t of the caller, or NULL for one
 * created for the call.  ws: logra_influence_stream_ws_size(Q, chunk_rows,
 * D, tr_dtype, topk) bytes (two staging buffers and one chunk's scoring
 * workspace).  SYNCHRONOUS: returns when the top-k is complete.
 * ---------------------------------------------------------------------- */
size_t logra_influence_stream_ws_size(int Q, int64_t chunk_rows, int D, int tr_dtype, int topk);
int logra_influence_stream(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q, const void *g_train_host,
                           int tr_dtype, int64_t ld_tr, int64_t N, int D, int64_t chunk_rows, int topk,
                           float *topk_val, int64_t *topk_idx, void *ws, size_t ws_bytes, void *stream,
                           void *copy_stream);

/* ------------------------------------------------------------------------
 * Out-of-core logging.  The projected gradients of every training example
 * are written to the store once, and the logging of the next batch overlaps
 * the saving of the current one (App. E.2, efficient data IO).
 *
 * logra_offload_rows: copies `rows` rows of `row_bytes` bytes from device
 * memory src (row stride ld_src bytes) to PINNED HOST memory dst
 * (hipHostMalloc; row stride ld_dst bytes), after the work already enqueued
 * on `stream` (an event recorded there is waited for on copy_stream; the
 * library keeps one such event per calling thread and device for the life of
 * the process), so the copy runs on copy_stream while the next batch is
 * projected on `stream`.
 * copy_stream NULL: the copy is enqueued on `stream` itself (in order, no
 * overlap on the device, still asynchronous for the host).  The copy is a
 * blit kernel: for a batch's rows on MI355X the in-order form is the cheaper
 * one (~20 us per 1 MB), as a concurrent blit shares the CUs with the
 * streaming projection.  done (optional, a hipEvent_t of the caller): recorded on the
 * copying stream after the copy; dst holds the rows once it has completed.
 * ASYNCHRONOUS.  src must not be overwritten until the copy has finished
 * (make `stream` wait for `done` before reusing those rows).
 * Errors: rows < 0, row_bytes <= 0 or a stride below row_bytes ->
 * INVALID_ARG; src (first and last row) not device memory or dst (first and
 * last row) not pinned host memory -> INVALID_ARG.  rows == 0: nothing.
 * ---------------------------------------------------------------------- */
int logra_offload_rows(const void *src, int64_t ld_src, void *dst, int64_t ld_dst, int64_t rows, int64_t row_bytes,
                       void *stream, void *copy_stream, void *done);

/* ------------------------------------------------------------------------
 * Store files.  At the paper's scale the store outgrows host memory as well
 * (Table 1: 3.5 TB); the paper keeps it on disk and overlaps reading it with
 * the influence computation (Sec. 4.2, Efficiency; App. E.2, efficient data
 * IO).  A store file holds rows of row_bytes bytes each, packed, from byte
 * file_offset of a file descriptor opened by the caller (the raw layout below
 * writes); row j starts at file_offset + j * row_bytes.  Reads and writes
 * go through the page cache (the streaming reader announces sequential access
 * with posix_fadvise).  Direct IO (O_DIRECT) is not usable here: the kernel
 * cannot pin pages of hipHostMalloc memory for it, and such reads fail with
 * EFAULT (LOGRA_ERR_IO).
 *
 * logra_store_read_rows / logra_store_write_rows: rows row0 .. row0+rows-1 of
 *   the file from / to host memory (rows at stride ld bytes), blocking, retried
 *   on interrupted and partial transfers.  A read past the end of the file
 *   returns LOGRA_ERR_IO.  No device memory is touched.
 *
 * logra_influence_stream_file: logra_influence_stream over a store file of N
 *   rows of D elements of tr_dtype (row_bytes = D * element size): a reader
 *   thread of the library reads chunk c + 1 into one of the two halves of
 *   host_buf while chunk c is copied to the device (copy_stream) and chunk
 *   c - 1 is scored (stream).  host_buf: PINNED host memory of at least
 *   2 * round_up(chunk_rows * row_bytes, 256) bytes.  ws: as for
 *   logra_influence_stream (logra_influence_stream_file_ws_size).  The top-k
 *   (global indices 0..N-1) is exactly that of logra_influence_scores over the
 *   whole store.  SYNCHRONOUS.  A failed or short read returns LOGRA_ERR_IO
 *   naming the chunk; the buffers are then idle.
 *
 * logra_offload_rows_file: write-behind of store rows.  `rows` device rows of
 *   row_bytes (stride ld_src bytes) are copied into host_buf (PINNED, packed,
 *   at least rows * row_bytes bytes) after the work on `stream`, as
 *   logra_offload_rows does, and a host function enqueued behind the copy on
 *   the same stream writes them to the file at file_offset (packed rows).
 *   ASYNCHRONOUS for the caller's thread: *io_status (host, may be NULL) is 1
 *   while pending, then LOGRA_OK or LOGRA_ERR_IO; `done` (optional hipEvent_t)
 *   is recorded after the write.  host_buf and io_status must stay valid, and
 *   host_buf unchanged, until the write has run (wait for `done`).
 * ---------------------------------------------------------------------- */
int logra_store_read_rows(int fd, int64_t file_offset, int64_t row0, int64_t rows, int64_t row_bytes, void *dst,
                          int64_t ld_dst);
int logra_store_write_rows(int fd, int64_t file_offset, int64_t row0, int64_t rows, int64_t row_bytes,
                           const void *src, int64_t ld_src);
size_t logra_influence_stream_file_ws_size(int Q, int64_t chunk_rows, int D, int tr_dtype, int topk);
int logra_influence_stream_file(const void *g_test_pre, int te_dtype, int64_t ld_te, int Q, int fd,
                                int64_t file_offset, int tr_dtype, int64_t N, int D, int64_t chunk_rows, int topk,
                                float *topk_val, int64_t *topk_idx, void *host_buf, size_t host_buf_bytes,
                                void *ws, size_t ws_bytes, void *stream, void *copy_stream);
int logra_offload_rows_file(const void *src, int64_t ld_src, int64_t rows, int64_t row_bytes, int fd,
                            int64_t file_offset, void *host_buf, size_t host_buf_bytes, int *io_status,
                            void *stream, void *copy_stream, void *done);

/* ------------------------------------------------------------------------
 * PCA initialisation of the projections (Sec. 3.2).  KFAC approximates a
 * layer's Hessian block by C_F (x) C_B, the Kronecker product of the
 * uncentered covariances of the layer's forward activations x and backward
 * output gradients dy; P_in and P_out are initialised with the top-k_in
 * eigenvectors of C_F and the top-k_out eigenvectors of C_B.
 *
 * logra_act_cov_accumulate: C[i][j] += sum over unmasked tokens (b, t) of
 *   a[b][t][i] * a[b][t][j]   (call it with x for C_F, with dy for C_B).
 *   a      device [B][T][n] of a_dtype (rows of n elements, contiguous);
 *          bf16: n a multiple of 8 (bf16 MFMA, fp32 accumulation); fp32: any n.
 *   mask   device u8 [B][T] or NULL (all tokens).  A masked token is never
 *          read, so NaN/Inf there cannot leak.
 *   C      device fp32 [n][n], accumulated in place and kept exactly
 *          symmetric (give it symmetric, e.g. zeroed).
 *   ws     workspace of logra_act_cov_ws_size(B, T) bytes (the list of
 *          non-empty 32-token slabs).  B = 0 or T = 0 is a no-op.
 * ---------------------------------------------------------------------- */
/* logra_act_cov_accumulate_group: the same for up to LOGRA_MAX_ACT_COV_GROUP
 *   factors of one batch in one launch, e.g. every KFAC factor of a
 *   transformer block (C_F of each distinct input, C_B of each layer).  The
 *   factors share B, T, the mask and a_dtype; each has its own activations a
 *   [B][T][n], n (same rule as above) and C [n][n].  No two C may overlap
 *   (LOGRA_ERR_INVALID_ARG); the same a may appear in several.  One tile pool
 *   over all factors, so a small factor no longer leaves most CUs idle.  Each
 *   C is identical to what logra_act_cov_accumulate gives it.  Workspace:
 *   logra_act_cov_ws_size(B, T), as for one factor.  n_desc above the maximum
 *   is LOGRA_ERR_UNSUPPORTED. */
#define LOGRA_MAX_ACT_COV_GROUP 32
typedef struct {
    const void *a;
    float *C;
    int n;
} logra_act_cov_desc;

size_t logra_act_cov_ws_size(int B, int T);
int logra_act_cov_accumulate_group(const logra_act_cov_desc *factors, int n_desc, int a_dtype, int B, int T,
                                   const uint8_t *mask, void *ws, size_t ws_bytes, void *stream);
int logra_act_cov_accumulate(const void *a, int a_dtype, int B, int T, int n, const uint8_t *mask, float *C,
                             void *ws, size_t ws_bytes, void *stream);

/* logra_pca_topk: the top-k eigenvectors of a symmetric PSD C (an
 * accumulated C_F or C_B) as the rows of a projection, P[e][i] = v_e[i] for
 * the eigenvalues in decreasing order, each v_e of unit norm and signed so
 * that its entry of largest magnitude (the lowest index among equal
 * magnitudes) is positive.
 *   C        device fp32 [n][n] (read only; only its symmetric part matters).
 *   k        1 <= k <= min(n, LOGRA_MAX_PCA_K).
 *   iters    >= 1 subspace iterations on p = min(n, max(2k, 16)) vectors,
 *            each one pass over C (fp32 MFMA products; fp64 orthonormalisation
 *            by shifted Cholesky-QR); then Rayleigh-Ritz with an fp64 Jacobi
 *            eigensolver.  The error of v_e falls like (theta_{p+1} /
 *            theta_e)^iters; 30 suits spectra whose top eigenvalues decay.
 *   P        device [k][ld_p] of P_dtype (F32 or BF16, rounded to nearest
 *            even), ld_p >= n.
 *   eigvals  device fp32 [k] (Ritz values) or NULL.
 *   ws       workspace of logra_pca_ws_size(n, k) bytes.
 * Asynchronous. */
#define LOGRA_MAX_PCA_K 64
size_t logra_pca_ws_size(int n, int k);
int logra_pca_topk(const float *C, int n, int k, int iters, void *P, int P_dtype, int64_t ld_p, float *eigvals,
                   void *ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* LOGRA_H */
