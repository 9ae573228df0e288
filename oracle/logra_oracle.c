/*
 * LoGra float64 CPU oracle -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * A plain, slow, obviously correct statement of what the LoGra hot path
 * computes (Choe et al., "What is Your Data Worth to GPT?", arXiv 2405.13954).
 * Every quantity is formed in double precision from the exact input bytes:
 * fp32 and bf16 inputs are widened to double without rounding, so the only
 * error left is the rounding of double-precision sums.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  It shares no code, header, table or constant with
 * the HIP implementation, and neither side includes the other.
 *
 * Conventions (the readings of the paper this file takes):
 *   - Arrays are row-major; the last index is contiguous.
 *   - A projected gradient G_b (k_out x k_in) is stored flattened as
 *     flat[o * k_in + i], the [out, in] shape of the bottleneck weight of the
 *     LoRA-like add-on (Sec. 3.1, Fig. 2).  Eq. (4)-(5) write vec() in the
 *     column-major order x_i (x) Dx_o; that is the permutation
 *     vec[i * k_out + o] of the same numbers.
 *   - A token contributes iff mask[b][t] != 0 (the attention mask passed to
 *     the logging context, App. B.1).  A masked token is never read, so its
 *     contribution is exactly zero even when its slots hold NaN or Inf.
 *   - The per-example gradient is a sum over tokens, not a mean (Eq. (4);
 *     the summed cross-entropy of App. B.1).
 *   - Dtype codes: 0 = fp32, 1 = bf16 (raw 16-bit patterns), 2 = fp64.
 *
 * Every loop is parallelised with OpenMP over an outer index only; inner
 * sums run in a fixed sequential order.
 */
#include <math.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_ERR_INVALID_ARG (-1)
#define OR_ERR_NOT_PD (-4)

#define OR_F32 0
#define OR_BF16 1
#define OR_F64 2

/* Exact widening of element i of an array of the given dtype.  A bf16
 * pattern is the upper half of an IEEE binary32 pattern, so shifting it into
 * place reproduces the value exactly. */
static double widen(const void *base, int dtype, int64_t i) {
    if (dtype == OR_F64) return ((const double *)base)[i];
    if (dtype == OR_F32) return (double)((const float *)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t *)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static int dtype_ok(int d) { return d == OR_F32 || d == OR_BF16 || d == OR_F64; }

/* ------------------------------------------------------------------------ */
/* Projection, factored form: the right-hand side of Eq. (5), Sec. 3.1.     */
/*   G_b = sum_t  (P_out Dx_{o,t}) (P_in x_{i,t})^T   over unmasked tokens.  */
/* Activations are projected first, then the outer product is accumulated;  */
/* the n_out x n_in gradient is never formed.                               */
/* x: [B][T][n_in], dy: [B][T][n_out], p_in: [k_in][n_in],                  */
/* p_out: [k_out][n_out] (all of dtype in_dtype); mask: [B][T] or NULL.     */
/* g: [B][k_out * k_in] doubles, overwritten.                               */
/* ------------------------------------------------------------------------ */
/* One example b of the factored projection; g_b (k_out * k_in doubles) is
 * overwritten.  Scratch: xp (k_in) and dp (k_out) doubles. */
static void project_example(const void *x, const void *dy, int in_dtype, int b, int T, int n_in,
                            int n_out, const uint8_t *mask, const void *p_in, const void *p_out,
                            int k_in, int k_out, double *gb, double *xp, double *dp) {
    int64_t D = (int64_t)k_in * k_out;
    for (int64_t d = 0; d < D; ++d) gb[d] = 0.0;
    for (int t = 0; t < T; ++t) {
        int64_t bt = (int64_t)b * T + t;
        if (mask && mask[bt] == 0) continue; /* masked: never read */
        /* x' = P_in x_t */
        for (int i = 0; i < k_in; ++i) {
            double s = 0.0;
            for (int j = 0; j < n_in; ++j)
                s += widen(p_in, in_dtype, (int64_t)i * n_in + j) * widen(x, in_dtype, bt * n_in + j);
            xp[i] = s;
        }
        /* dy' = P_out Dx_{o,t} */
        for (int o = 0; o < k_out; ++o) {
            double s = 0.0;
            for (int j = 0; j < n_out; ++j)
                s += widen(p_out, in_dtype, (int64_t)o * n_out + j) * widen(dy, in_dtype, bt * n_out + j);
            dp[o] = s;
        }
        /* outer product dy' x'^T, accumulated over tokens */
        for (int o = 0; o < k_out; ++o)
            for (int i = 0; i < k_in; ++i) gb[(int64_t)o * k_in + i] += dp[o] * xp[i];
    }
}

int oracle_project_factored(const void *x, const void *dy, int in_dtype, int B, int T,
                            int n_in, int n_out, const uint8_t *mask, const void *p_in,
                            const void *p_out, int k_in, int k_out, double *g) {
    if (B < 0 || T < 0 || n_in <= 0 || n_out <= 0 || k_in <= 0 || k_out <= 0) return OR_ERR_INVALID_ARG;
    if (!dtype_ok(in_dtype)) return OR_ERR_INVALID_ARG;
    int64_t D = (int64_t)k_in * k_out;
#pragma omp parallel for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        double *xp = (double *)malloc(sizeof(double) * (size_t)k_in);
        double *dp = (double *)malloc(sizeof(double) * (size_t)k_out);
        project_example(x, dy, in_dtype, b, T, n_in, n_out, mask, p_in, p_out, k_in, k_out, g + (int64_t)b * D,
                        xp, dp);
        free(xp);
        free(dp);
    }
    return OR_OK;
}

/* The same projection for n_layers layers of one batch (shared B, T, mask,
 * k_in, k_out, dtype; layer l has its own tensors, widths and output
 * g[l], [B][k_out * k_in]).  Each (layer, example) is computed exactly as
 * above; only the parallel loop runs over the pairs. */
int oracle_project_factored_layers(int n_layers, const void *const *x, const void *const *dy, int in_dtype,
                                   int B, int T, const int *n_in, const int *n_out, const uint8_t *mask,
                                   const void *const *p_in, const void *const *p_out, int k_in, int k_out,
                                   double *const *g) {
    if (n_layers < 0 || B < 0 || T < 0 || k_in <= 0 || k_out <= 0 || !dtype_ok(in_dtype))
        return OR_ERR_INVALID_ARG;
    for (int l = 0; l < n_layers; ++l)
        if (n_in[l] <= 0 || n_out[l] <= 0) return OR_ERR_INVALID_ARG;
    int64_t D = (int64_t)k_in * k_out;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int l = 0; l < n_layers; ++l)
        for (int b = 0; b < B; ++b) {
            double *xp = (double *)malloc(sizeof(double) * (size_t)k_in);
            double *dp = (double *)malloc(sizeof(double) * (size_t)k_out);
            project_example(x[l], dy[l], in_dtype, b, T, n_in[l], n_out[l], mask, p_in[l], p_out[l], k_in, k_out,
                            g[l] + (int64_t)b * D, xp, dp);
            free(xp);
            free(dp);
        }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Projection, from the full per-example gradient: Eq. (4) then the left    */
/* side of Eq. (5).  DW_b = sum_t Dx_{o,t} x_{i,t}^T (n_out x n_in), then   */
/* G_b = P_out DW_b P_in^T.  Materialises DW, so small inputs only; it      */
/* exists to pin the factored form above.  Same arguments and output.       */
/* ------------------------------------------------------------------------ */
int oracle_project_dense(const void *x, const void *dy, int in_dtype, int B, int T, int n_in,
                         int n_out, const uint8_t *mask, const void *p_in, const void *p_out,
                         int k_in, int k_out, double *g) {
    if (B < 0 || T < 0 || n_in <= 0 || n_out <= 0 || k_in <= 0 || k_out <= 0) return OR_ERR_INVALID_ARG;
    if (!dtype_ok(in_dtype)) return OR_ERR_INVALID_ARG;
    int64_t D = (int64_t)k_in * k_out;
#pragma omp parallel for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        double *dw = (double *)calloc((size_t)n_out * (size_t)n_in, sizeof(double));
        double *tmp = (double *)malloc(sizeof(double) * (size_t)k_out * (size_t)n_in);
        /* Eq. (4): the weight gradient is a sum over tokens of outer products */
        for (int t = 0; t < T; ++t) {
            int64_t bt = (int64_t)b * T + t;
            if (mask && mask[bt] == 0) continue;
            for (int a = 0; a < n_out; ++a) {
                double d = widen(dy, in_dtype, bt * n_out + a);
                for (int c = 0; c < n_in; ++c)
                    dw[(int64_t)a * n_in + c] += d * widen(x, in_dtype, bt * n_in + c);
            }
        }
        /* tmp = P_out DW  (k_out x n_in) */
        for (int o = 0; o < k_out; ++o)
            for (int c = 0; c < n_in; ++c) {
                double s = 0.0;
                for (int a = 0; a < n_out; ++a)
                    s += widen(p_out, in_dtype, (int64_t)o * n_out + a) * dw[(int64_t)a * n_in + c];
                tmp[(int64_t)o * n_in + c] = s;
            }
        /* G = tmp P_in^T  (k_out x k_in) */
        double *gb = g + (int64_t)b * D;
        for (int o = 0; o < k_out; ++o)
            for (int i = 0; i < k_in; ++i) {
                double s = 0.0;
                for (int c = 0; c < n_in; ++c)
                    s += tmp[(int64_t)o * n_in + c] * widen(p_in, in_dtype, (int64_t)i * n_in + c);
                gb[(int64_t)o * k_in + i] = s;
            }
        free(dw);
        free(tmp);
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Covariance of projected gradients: the empirical Fisher of Assumption 1  */
/* (App. D), used as the projected Hessian P H P^T of Eq. (3), Sec. 2.      */
/*   S[d][e] += sum_b g_b[d] g_b[e]    (unnormalised; caller tracks N)      */
/* g: B rows of D elements at row stride ld (elements), dtype g_dtype.      */
/* S: [D][D] doubles, accumulated in place.                                 */
/* ------------------------------------------------------------------------ */
int oracle_cov_accumulate(const void *g, int g_dtype, int64_t ld, int B, int D, double *S) {
    if (B < 0 || D <= 0 || ld < D || !dtype_ok(g_dtype)) return OR_ERR_INVALID_ARG;
#pragma omp parallel for schedule(dynamic, 4)
    for (int d = 0; d < D; ++d)
        for (int e = 0; e < D; ++e) {
            double s = 0.0;
            for (int b = 0; b < B; ++b)
                s += widen(g, g_dtype, (int64_t)b * ld + d) * widen(g, g_dtype, (int64_t)b * ld + e);
            S[(int64_t)d * D + e] += s;
        }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Damped inverse applied to test gradients: step (1) of the influence      */
/* function (iHVP with g_te, Sec. 2 after Eq. (2)), in the projected space  */
/* of Eq. (3), for one layer block.                                         */
/*   C = S / N                          (empirical Fisher, App. D)          */
/*   lambda = r * tr(C) / D             (r x mean eigenvalue, App. C;       */
/*                                       the mean of the eigenvalues of a   */
/*                                       symmetric matrix is its trace / D) */
/*   out_q = (C + lambda I)^{-1} g_q    (Cholesky, forward and back solve)  */
/* r < 0 selects the identity preconditioner: out = g.                      */
/* S: [D][D] doubles (only the lower triangle is read).                     */
/* g: Q rows at stride ld_g, dtype g_dtype; out: Q rows at stride ld_out.   */
/* lambda_out (may be NULL) receives lambda.  Returns OR_ERR_NOT_PD if a    */
/* pivot of the factorisation is not positive.                              */
/* ------------------------------------------------------------------------ */
int oracle_precondition(const double *S, int D, int64_t N, double r, const void *g, int g_dtype,
                        int64_t ld_g, int Q, double *out, int64_t ld_out, double *lambda_out) {
    if (D <= 0 || Q < 0 || ld_g < D || ld_out < D || !dtype_ok(g_dtype)) return OR_ERR_INVALID_ARG;
    if (r < 0.0) {
        for (int q = 0; q < Q; ++q)
            for (int d = 0; d < D; ++d)
                out[(int64_t)q * ld_out + d] = widen(g, g_dtype, (int64_t)q * ld_g + d);
        if (lambda_out) *lambda_out = 0.0;
        return OR_OK;
    }
    if (N <= 0) return OR_ERR_INVALID_ARG;
    double *L = (double *)calloc((size_t)D * (size_t)D, sizeof(double));
    double tr = 0.0;
    for (int d = 0; d < D; ++d) tr += S[(int64_t)d * D + d] / (double)N;
    double lambda = r * tr / (double)D;
    if (lambda_out) *lambda_out = lambda;
    /* Cholesky-Banachiewicz, row by row: A = C + lambda I = L L^T */
    for (int i = 0; i < D; ++i) {
        for (int j = 0; j <= i; ++j) {
            double a = S[(int64_t)i * D + j] / (double)N + (i == j ? lambda : 0.0);
            double s = 0.0;
            for (int m = 0; m < j; ++m) s += L[(int64_t)i * D + m] * L[(int64_t)j * D + m];
            if (i == j) {
                double piv = a - s;
                if (!(piv > 0.0)) {
                    free(L);
                    return OR_ERR_NOT_PD;
                }
                L[(int64_t)i * D + i] = sqrt(piv);
            } else {
                L[(int64_t)i * D + j] = (a - s) / L[(int64_t)j * D + j];
            }
        }
    }
#pragma omp parallel for schedule(dynamic, 1)
    for (int q = 0; q < Q; ++q) {
        double *z = out + (int64_t)q * ld_out;
        /* forward: L y = g */
        for (int i = 0; i < D; ++i) {
            double s = widen(g, g_dtype, (int64_t)q * ld_g + i);
            for (int m = 0; m < i; ++m) s -= L[(int64_t)i * D + m] * z[m];
            z[i] = s / L[(int64_t)i * D + i];
        }
        /* backward: L^T z = y */
        for (int i = D - 1; i >= 0; --i) {
            double s = z[i];
            for (int m = i + 1; m < D; ++m) s -= L[(int64_t)m * D + i] * z[m];
            z[i] = s / L[(int64_t)i * D + i];
        }
    }
    free(L);
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Influence scores: step (2) of the influence function (Sec. 2, Eq. (2)),  */
/* the dot product of each preconditioned test gradient with each stored    */
/* train gradient, in the projected space of Eq. (3).  With a block-diagonal */
/* (per-layer) Hessian the whole-model score is the dot product over the    */
/* concatenated layer blocks.                                               */
/*   s[q][j] = sum_d te[q][d] * tr[j][d]                                    */
/* ------------------------------------------------------------------------ */
int oracle_scores(const void *te, int te_dtype, int64_t ld_te, int Q, const void *tr,
                  int tr_dtype, int64_t ld_tr, int64_t N, int D, double *s, int64_t ld_s) {
    if (Q < 0 || N < 0 || D <= 0 || ld_te < D || ld_tr < D || ld_s < N) return OR_ERR_INVALID_ARG;
    if (!dtype_ok(te_dtype) || !dtype_ok(tr_dtype)) return OR_ERR_INVALID_ARG;
#pragma omp parallel for schedule(dynamic, 64) collapse(2)
    for (int q = 0; q < Q; ++q)
        for (int64_t j = 0; j < N; ++j) {
            double acc = 0.0;
            for (int d = 0; d < D; ++d)
                acc += widen(te, te_dtype, (int64_t)q * ld_te + d) * widen(tr, tr_dtype, j * ld_tr + d);
            s[(int64_t)q * ld_s + j] = acc;
        }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Self-influence of a gradient (the normaliser of l-RelatIF, Sec. 4.2,     */
/* which divides each influence score by the training example's own         */
/* influence to penalise large-gradient outliers):                          */
/*   self_j = g_j^T (C + lambda I)^{-1} g_j                                 */
/* for one layer block, with C, lambda as in oracle_precondition (the       */
/* whole-model value of a block-diagonal Hessian is the sum over blocks).   */
/* Written as its definition: the damped inverse applied to g_j, then the   */
/* dot product with g_j.                                                    */
/* ------------------------------------------------------------------------ */
int oracle_self_influence(const double *S, int D, int64_t N, double r, const void *g, int g_dtype,
                          int64_t ld_g, int rows, double *self_out) {
    if (D <= 0 || rows < 0 || ld_g < D || !dtype_ok(g_dtype)) return OR_ERR_INVALID_ARG;
    double *y = (double *)malloc((size_t)(rows > 0 ? rows : 1) * (size_t)D * sizeof(double));
    const int rc = oracle_precondition(S, D, N, r, g, g_dtype, ld_g, rows, y, D, NULL);
    if (rc != OR_OK) {
        free(y);
        return rc;
    }
#pragma omp parallel for schedule(static)
    for (int j = 0; j < rows; ++j) {
        double acc = 0.0;
        for (int d = 0; d < D; ++d) acc += widen(g, g_dtype, (int64_t)j * ld_g + d) * y[(int64_t)j * D + d];
        self_out[j] = acc;
    }
    free(y);
    return OR_OK;
}

/* Normalised scores: s[q][j] / sqrt(self_tr[j]) (l-RelatIF), and also       */
/* / sqrt(self_te[q]) when self_te is given (the cosine form: the cosine of  */
/* the angle between the two gradients in the (C + lambda I)^{-1} inner      */
/* product).  A zero self-influence (a zero gradient, whose raw scores are   */
/* zero) gives a zero normalised score.                                      */
int oracle_normalise_scores(double *s, int64_t ld_s, int Q, int64_t N, const double *self_te,
                            const double *self_tr) {
    if (Q < 0 || N < 0 || ld_s < N || !self_tr) return OR_ERR_INVALID_ARG;
    for (int q = 0; q < Q; ++q)
        for (int64_t j = 0; j < N; ++j) {
            double den = self_tr[j];
            if (self_te) den *= self_te[q];
            s[(int64_t)q * ld_s + j] = den > 0.0 ? s[(int64_t)q * ld_s + j] / sqrt(den) : 0.0;
        }
    return OR_OK;
}

/* ------------------------------------------------------------------------ */
/* Uncentered activation covariance of one layer, the KFAC factor behind     */
/* the PCA initialisation of the projections (Sec. 3.2: C_F from the forward */
/* activations x, C_B from the backward output gradients Dx_o, H_KFAC =      */
/* C_F (x) C_B; P_i and P_o are their top-k eigenvectors):                   */
/*   C[i][j] += sum over unmasked (b, t) of a_bt[i] a_bt[j]                  */
/* a: [B][T][n] of dtype a_dtype; mask: [B][T] or NULL (NULL = all tokens);  */
/* a masked token is never read.  C: [n][n] doubles, accumulated in place.   */
/* ------------------------------------------------------------------------ */
int oracle_act_cov(const void *a, int a_dtype, int B, int T, int n, const uint8_t *mask, double *C) {
    if (B < 0 || T < 0 || n <= 0 || !dtype_ok(a_dtype)) return OR_ERR_INVALID_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < n; ++i)
        for (int b = 0; b < B; ++b)
            for (int t = 0; t < T; ++t) {
                int64_t bt = (int64_t)b * T + t;
                if (mask && mask[bt] == 0) continue;
                double ai = widen(a, a_dtype, bt * n + i);
                for (int j = 0; j < n; ++j) C[(int64_t)i * n + j] += ai * widen(a, a_dtype, bt * n + j);
            }
    return OR_OK;
}

/* (value, index) a ranks before (value, index) b: larger value first, the   */
/* lower train index on equal values.  Padding (index -1) ranks last.        */
static int ranks_before(double va, int64_t ia, double vb, int64_t ib) {
    if (ia < 0) return 0;
    if (ib < 0) return 1;
    if (va != vb) return va > vb;
    return ia < ib;
}

/* ------------------------------------------------------------------------ */
/* Per-query top-k of the most valuable training data (Sec. 4.1, App. A):   */
/* the k largest signed scores of each row, ties to the lower train index.  */
/* s: [Q][N] at row stride ld_s; train row j has global index base + j.     */
/* val/idx: [Q][k]; slots beyond the number of candidates hold              */
/* (-inf, -1).  Kept sorted by insertion into a k-long ranked list.         */
/* ------------------------------------------------------------------------ */
int oracle_topk(const double *s, int64_t ld_s, int Q, int64_t N, int64_t base, int k,
                double *val, int64_t *idx) {
    if (Q < 0 || N < 0 || k <= 0 || ld_s < N) return OR_ERR_INVALID_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int q = 0; q < Q; ++q) {
        double *v = val + (int64_t)q * k;
        int64_t *ix = idx + (int64_t)q * k;
        for (int r = 0; r < k; ++r) {
            v[r] = -INFINITY;
            ix[r] = -1;
        }
        for (int64_t j = 0; j < N; ++j) {
            double sj = s[(int64_t)q * ld_s + j];
            int64_t gj = base + j;
            if (!ranks_before(sj, gj, v[k - 1], ix[k - 1])) continue;
            int r = k - 1;
            while (r > 0 && ranks_before(sj, gj, v[r - 1], ix[r - 1])) {
                v[r] = v[r - 1];
                ix[r] = ix[r - 1];
                --r;
            }
            v[r] = sj;
            ix[r] = gj;
        }
    }
    return OR_OK;
}

/* Number of OpenMP threads a parallel region of this library uses. */
int oracle_num_threads(void) {
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
