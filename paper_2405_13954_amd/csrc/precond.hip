// Damped inverse applied to test gradients, per layer block (the iHVP step of
// the influence function, Sec. 2 Eq. (2), in the projected space of Eq. (3)):
//
//   C = S / N,  lambda = r * tr(C) / D   (r x mean eigenvalue, App. C)
//   out_q = (C + lambda I)^{-1} g_q
//
// All arithmetic is float64; S may be given in fp32 or fp64.  Steps, each batched over layer blocks
// (blockIdx.y):
//   1. lambda per block (fixed-order tree sum of the diagonal);
//   2. A = S/N + lambda I into the workspace (lower triangle);
//   3. blocked right-looking Cholesky, 64-wide panels: factor the diagonal
//      block in LDS, solve the panel below it, SYRK-update the trailing
//      matrix;  a non-positive pivot sets the block's status word;
//   4. the inverse of each 64x64 diagonal tile of L;
//   5. blocked forward and backward substitution for 64 right-hand sides per
//      workgroup, every step a 64x64x64 product on the fp64 matrix cores:
//        forward   R_i = G_i - sum_{j<i} L_ij Y_j,     Y_i = inv(L_ii) R_i
//        backward  R_i = Y_i - sum_{j>i} L_ji^T Z_j,   Z_i = inv(L_ii)^T R_i
//      (tiles staged through LDS with coalesced loads, Y and Z in the
//      workspace), so no step is a row-by-row recurrence.
#include "common.h"
#include "internal.h"

namespace logra {
namespace {

constexpr int NB = 64;   // panel width / tile edge
constexpr int LT = NB + 1;

struct WsLayout {
    double *A;      // [n_blocks][D][D], lower triangle: C + lambda I, then L
    double *lam;    // [n_blocks]
    int *info;      // [n_blocks] 0 or 1 + first non-positive pivot
    double *Linv;   // [n_blocks][nbt][64][64] inverses of the diagonal tiles of L
    double *Y;      // [n_blocks][D][Qp] forward solutions
    double *Z;      // [n_blocks][D][Qp] backward solutions
};

inline int tiles_of(int D) { return (D + NB - 1) / NB; }
inline int padded_q(int Q) { return (Q + NB - 1) / NB * NB; }

inline WsLayout ws_layout(void *ws, int D, int n_blocks, int Q) {
    char *p = static_cast<char *>(ws);
    const size_t nb = static_cast<size_t>(n_blocks);
    WsLayout w;
    w.A = reinterpret_cast<double *>(p);
    p += align256(sizeof(double) * nb * D * D);
    w.lam = reinterpret_cast<double *>(p);
    p += align256(sizeof(double) * nb);
    w.info = reinterpret_cast<int *>(p);
    p += align256(sizeof(int) * nb);
    w.Linv = reinterpret_cast<double *>(p);
    p += align256(sizeof(double) * nb * tiles_of(D) * NB * NB);
    w.Y = reinterpret_cast<double *>(p);
    p += align256(sizeof(double) * nb * D * padded_q(Q));
    w.Z = reinterpret_cast<double *>(p);
    return w;
}

template <typename TS>
__global__ __launch_bounds__(256) void k_lambda(const TS *S, int D, int64_t N, double r,
                                                double *lam) {
    __shared__ double part[256];
    const int blk = blockIdx.x;
    const TS *Sb = S + static_cast<size_t>(blk) * D * D;
    double s = 0.0;
    for (int d = threadIdx.x; d < D; d += 256) s += load_in_d<TS>(Sb + static_cast<size_t>(d) * D + d);
    part[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) lam[blk] = r * (part[0] / static_cast<double>(N)) / static_cast<double>(D);
}

template <typename TS>
__global__ __launch_bounds__(256) void k_form(const TS *S, int D, int64_t N, const double *lam,
                                              double *A, int *info) {
    const int blk = blockIdx.y, i = blockIdx.x;
    const TS *Sr = S + (static_cast<size_t>(blk) * D + i) * D;
    double *Ar = A + (static_cast<size_t>(blk) * D + i) * D;
    const double inv = 1.0 / static_cast<double>(N);
    for (int j = threadIdx.x; j <= i; j += 256) {
        double v = load_in_d<TS>(Sr + j) * inv;
        if (j == i) v += lam[blk];
        Ar[j] = v;
    }
    if (i == 0 && threadIdx.x == 0) info[blk] = 0;
}

// Unblocked Cholesky of the nb x nb diagonal block at (k0, k0); one wave.
// Lane t holds row t in registers; at step j the pivot and then column j of
// the rows below come from their lanes by readlane, so no step needs LDS or
// a barrier.  Each row's update A_tk -= L_tj L_kj is the same fused operation
// in the same order as a textbook right-looking factorisation.  Entries above
// the diagonal collect meaningless values and are never read; rows past nb
// are identity rows, so every step runs (unit pivots there).
__global__ __launch_bounds__(64) void k_potrf_diag(double *A_all, int D, int k0, int *info) {
    __shared__ double a[NB * LT];
    const int blk = blockIdx.x, t = threadIdx.x;
    double *A = A_all + static_cast<size_t>(blk) * D * D;
    const int nb = min(NB, D - k0);
    for (int i = 0; i < nb; ++i)
        if (t <= i) a[i * LT + t] = A[static_cast<size_t>(k0 + i) * D + k0 + t];
    __syncthreads();
    double r[NB];
    const int tl = t < nb ? t : nb - 1;   // clamped: every lane reads, padding is selected afterwards
#pragma unroll
    for (int k = 0; k < NB; ++k) {
        const double v = a[tl * LT + (k < tl ? k : tl)];
        r[k] = t < nb ? (k <= t ? v : 0.0) : (k == t ? 1.0 : 0.0);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        double piv = readlane_d(r[j], j);
        if (!(piv > 0.0)) {
            if (t == 0 && info[blk] == 0) info[blk] = k0 + j + 1;
            piv = 1.0;   // keep going; the result is reported as not PD
        }
        const double d = sqrt(piv);
        r[j] = t == j ? d : t > j ? r[j] / d : r[j];
#pragma unroll
        for (int k = j + 1; k < NB; ++k) {
            r[k] = fma(-r[j], readlane_d(r[j], k), r[k]);
            if ((k - j) % 8 == 0) __builtin_amdgcn_sched_barrier(0);   // at most 8 readlane pairs live
        }
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int k = 0; k < NB; ++k)
        if (k <= t) a[t * LT + k] = r[k];
    __syncthreads();
    for (int i = 0; i < nb; ++i)
        if (t <= i) A[static_cast<size_t>(k0 + i) * D + k0 + t] = a[i * LT + t];
}

// Forward substitution L x = b for one right-hand side per lane, x in
// registers (b on entry), L the lower-triangular 64 x 64 tile in LDS (row
// stride LT; past the valid rows an identity), read at wave-uniform
// addresses so that every read is a broadcast: x_j = x_j / L_jj, then
// x_k -= L_kj x_j for k > j.
__device__ __forceinline__ void fwd_subst(double (&x)[NB], const double *l) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        x[j] = x[j] / l[j * LT + j];
#pragma unroll
        for (int k = j + 1; k < NB; ++k) {
            x[k] = fma(-l[k * LT + j], x[j], x[k]);
            if ((k - j) % 8 == 0) __builtin_amdgcn_sched_barrier(0);   // at most 8 broadcast reads live
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Rows below the diagonal block: L21 = A21 L11^{-T}; one row per lane.
__global__ __launch_bounds__(64) void k_trsm_panel(double *A_all, int D, int k0) {
    __shared__ double l11[NB * LT];
    __shared__ double x[NB * LT];
    const int blk = blockIdx.y, t = threadIdx.x;
    double *A = A_all + static_cast<size_t>(blk) * D * D;
    const int nb = min(NB, D - k0);
    const int r0 = k0 + nb + blockIdx.x * NB;
    const int nr = min(NB, D - r0);
    for (int i = 0; i < NB; ++i)   // identity past nb
        l11[i * LT + t] = i < nb ? (t <= i ? A[static_cast<size_t>(k0 + i) * D + k0 + t] : 0.0) : (t == i ? 1.0 : 0.0);
    for (int i = 0; i < nr; ++i) x[i * LT + t] = (t < nb) ? A[static_cast<size_t>(r0 + i) * D + k0 + t] : 0.0;
    __syncthreads();
    // row t solves x L11^T = a, i.e. L11 x^T = a^T
    double r[NB];
#pragma unroll
    for (int k = 0; k < NB; ++k) r[k] = t < nr ? x[t * LT + k] : 0.0;
    fwd_subst(r, l11);
#pragma unroll
    for (int k = 0; k < NB; ++k) x[t * LT + k] = r[k];   // each lane rewrites only its own row
    __syncthreads();
    for (int i = 0; i < nr; ++i)
        if (t < nb) A[static_cast<size_t>(r0 + i) * D + k0 + t] = x[i * LT + t];
}

// Trailing update A22 -= L21 L21^T on lower-triangle 64x64 tiles.
__global__ __launch_bounds__(256) void k_syrk_update(double *A_all, int D, int k0, int nt) {
    __shared__ double li[NB * LT];
    __shared__ double lj[NB * LT];
    const int blk = blockIdx.y;
    double *A = A_all + static_cast<size_t>(blk) * D * D;
    const int nb = min(NB, D - k0);
    const int base = k0 + nb;
    // tile t -> (ti >= tj), enumerated row by row of the lower triangle
    int t = blockIdx.x, ti = 0;
    while (t > ti) {
        t -= ti + 1;
        ++ti;
    }
    const int tj = t;
    const int I = base + ti * NB, J = base + tj * NB;
    const int tid = threadIdx.x;
    for (int e = tid; e < NB * NB; e += 256) {
        const int r = e / NB, c = e - (e / NB) * NB;
        li[r * LT + c] = (I + r < D && c < nb) ? A[static_cast<size_t>(I + r) * D + k0 + c] : 0.0;
        lj[r * LT + c] = (J + r < D && c < nb) ? A[static_cast<size_t>(J + r) * D + k0 + c] : 0.0;
    }
    __syncthreads();
    const int ta = tid >> 4, tb = tid & 15;
    double acc[4][4] = {};
    for (int m = 0; m < nb; ++m) {
        double a[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            a[u] = li[(4 * ta + u) * LT + m];
            b[u] = lj[(4 * tb + u) * LT + m];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[u][v] = fma(a[u], b[v], acc[u][v]);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int i = I + 4 * ta + u;
        if (i >= D) break;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = J + 4 * tb + v;
            if (j <= i) A[static_cast<size_t>(i) * D + j] -= acc[u][v];
        }
    }
}

// Inverse of the lower-triangular 64x64 diagonal tile t of L (zero padded
// past D): lane c solves L_tt w = e_c in registers, giving column c.
__global__ __launch_bounds__(64) void k_diag_inv(const double *A_all, int D, double *Linv_all) {
    __shared__ double a[NB * LT];
    const int t = blockIdx.x, blk = blockIdx.y, c = threadIdx.x;
    const double *A = A_all + static_cast<size_t>(blk) * D * D;
    const int r0 = t * NB, nb = min(NB, D - r0);
    for (int i = 0; i < NB; ++i)   // identity past nb
        a[i * LT + c] = i < nb ? (c <= i ? A[static_cast<size_t>(r0 + i) * D + r0 + c] : 0.0) : (c == i ? 1.0 : 0.0);
    __syncthreads();
    double w[NB];   // e_c for the valid columns; padded columns of the inverse are zero
#pragma unroll
    for (int k = 0; k < NB; ++k) w[k] = (k == c && c < nb) ? 1.0 : 0.0;
    fwd_subst(w, a);
    double *W = Linv_all + (static_cast<size_t>(blk) * gridDim.x + t) * NB * NB;
#pragma unroll
    for (int r = 0; r < NB; ++r) W[r * NB + c] = w[r];
}

// Blocked substitution on the matrix cores for 64 right-hand sides (queries
// q0 .. q0+63) of one layer block.  Wave w owns rows 16w..16w+15 of the
// 64 x 64 (rows x queries) tile; acc[c] holds columns 16c..16c+15 in the
// fp64 16x16 result layout (register r of lane l: row l/16 + 4r).
// IDENT: the right-hand sides are the identity columns (g is not read) and
// only the forward solve runs, leaving L^{-1} in Y.
template <typename TIn, typename TOut, bool IDENT = false>
__global__ __launch_bounds__(256) void k_trsm_f64(const double *A_all, const double *Linv_all, int D,
                                                  const TIn *g, int64_t ld_in, int Q, int Qp, double *Y_all,
                                                  double *Z_all, TOut *out, int64_t ld_out) {
    __shared__ double La[NB * LT];   // A operand tile [row][k]
    __shared__ double Yb[NB * LT];   // B operand tile [k][query]
    const int blk = blockIdx.y, q0 = blockIdx.x * NB;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int row = lane & 15, kg = lane >> 4;
    const int nbt = (D + NB - 1) / NB;
    const double *L = A_all + static_cast<size_t>(blk) * D * D;
    const double *Li = Linv_all + static_cast<size_t>(blk) * nbt * NB * NB;
    double *Y = Y_all + static_cast<size_t>(blk) * D * Qp;
    double *Z = Z_all + static_cast<size_t>(blk) * D * Qp;
    f64x4 acc[4];

    // Tile staging: each thread's 16 elements are loaded into registers first
    // (all loads in flight), then stored to LDS.
    constexpr int kPer = NB * NB / 256;
    // La[rr][cc] = L[r0+rr][c0+cc] (strictly lower tiles only), or its transpose.
    auto stage_L = [&](int r0, int c0, bool transpose) {
        double v[kPer];
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int e = tid + 256 * q;
            const int u = e / NB, w2 = e - (e / NB) * NB;   // consecutive threads: consecutive w2
            const int rr = transpose ? c0 + u : r0 + u, cc = transpose ? r0 + w2 : c0 + w2;
            v[q] = (rr < D && cc < D) ? L[static_cast<size_t>(rr) * D + cc] : 0.0;
        }
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int e = tid + 256 * q;
            const int u = e / NB, w2 = e - (e / NB) * NB;
            if (!transpose) La[u * LT + w2] = v[q];
            else La[w2 * LT + u] = v[q];   // La[w2][u] = L[c0+u][r0+w2]
        }
    };
    auto stage_Linv = [&](int i, bool transpose) {
        const double *T = Li + static_cast<size_t>(i) * NB * NB;
        double v[kPer];
#pragma unroll
        for (int q = 0; q < kPer; ++q) v[q] = T[tid + 256 * q];
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int e = tid + 256 * q;
            const int u = e / NB, w2 = e - (e / NB) * NB;
            if (!transpose) La[u * LT + w2] = v[q];
            else La[w2 * LT + u] = v[q];
        }
    };
    auto stage_B = [&](const double *src, int j) {   // Yb[kk][qq] = src[j*64 + kk][q0 + qq]
        double v[kPer];
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int e = tid + 256 * q;
            const int kk = e / NB, qq = e - (e / NB) * NB;
            v[q] = (j * NB + kk < D) ? src[static_cast<size_t>(j * NB + kk) * Qp + q0 + qq] : 0.0;
        }
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int e = tid + 256 * q;
            const int kk = e / NB, qq = e - (e / NB) * NB;
            Yb[kk * LT + qq] = v[q];
        }
    };
    auto mma = [&](double sign) {
#pragma unroll 4
        for (int s4 = 0; s4 < NB / 4; ++s4) {
            const double a = sign * La[(16 * w + row) * LT + 4 * s4 + kg];
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[c] = mfma16_f64(a, Yb[(4 * s4 + kg) * LT + 16 * c + row], acc[c]);
        }
    };
    auto acc_to_B = [&]() {
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int r = 0; r < 4; ++r) Yb[(16 * w + kg + 4 * r) * LT + 16 * c + row] = acc[c][r];
    };
    auto zero = [&]() {
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = f64x4{0.0, 0.0, 0.0, 0.0};
    };
    auto store_ws = [&](double *dst, int i) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int d = i * NB + 16 * w + kg + 4 * r;
                if (d < D) dst[static_cast<size_t>(d) * Qp + q0 + 16 * c + row] = acc[c][r];
            }
    };

    // ---------------- forward: L Y = G ----------------
    for (int i = 0; i < nbt; ++i) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int q = q0 + 16 * c + row, d = i * NB + 16 * w + kg + 4 * r;
                if (IDENT)
                    acc[c][r] = (q < Q && d == q) ? 1.0 : 0.0;
                else
                    acc[c][r] = (q < Q && d < D) ? load_in_d<TIn>(g + static_cast<int64_t>(q) * ld_in +
                                                                   static_cast<int64_t>(blk) * D + d)
                                                 : 0.0;
            }
        for (int j = 0; j < i; ++j) {
            stage_L(i * NB, j * NB, false);
            stage_B(Y, j);
            __syncthreads();
            mma(-1.0);
            __syncthreads();
        }
        acc_to_B();
        stage_Linv(i, false);
        __syncthreads();
        zero();
        mma(1.0);
        store_ws(Y, i);
        __syncthreads();
    }
    if (IDENT) return;
    // ---------------- backward: L^T Z = Y ----------------
    for (int i = nbt - 1; i >= 0; --i) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int d = i * NB + 16 * w + kg + 4 * r;
                acc[c][r] = d < D ? Y[static_cast<size_t>(d) * Qp + q0 + 16 * c + row] : 0.0;
            }
        for (int j = i + 1; j < nbt; ++j) {
            stage_L(i * NB, j * NB, true);
            stage_B(Z, j);
            __syncthreads();
            mma(-1.0);
            __syncthreads();
        }
        acc_to_B();
        stage_Linv(i, true);
        __syncthreads();
        zero();
        mma(1.0);
        store_ws(Z, i);
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int q = q0 + 16 * c + row, d = i * NB + 16 * w + kg + 4 * r;
                if (q < Q && d < D)
                    store_out_d<TOut>(out + static_cast<int64_t>(q) * ld_out + static_cast<int64_t>(blk) * D + d,
                                      acc[c][r]);
            }
        __syncthreads();
    }
}

__global__ __launch_bounds__(256) void k_clear_info(int *info, int n) {
    for (int i = threadIdx.x; i < n; i += 256) info[i] = 0;
}

// W = L^{-1} (fp64, rows d, columns q of the forward solution) as two bf16
// arrays whose sum carries about 16 significant bits: hi = RNE(W), lo =
// RNE(W - hi); rows d past D (up to Dp = gridDim.x) are zero.  Split layout:
// hi [blk][Dp][D] then lo; interleaved: [blk][Dp][2D], the 64 columns of
// chunk c at 128 c (hi) and 128 c + 64 (lo).  With `ident`, W = I.
__global__ __launch_bounds__(256) void k_split_w(const double *Y_all, int D, int Qp, bool ident,
                                                  bool interleaved, bf16_bits *w_hi, bf16_bits *w_lo) {
    const int blk = blockIdx.y, d = blockIdx.x;
    const size_t row = static_cast<size_t>(blk) * gridDim.x + d;
    bf16_bits *h = interleaved ? w_hi + row * 2 * D : w_hi + row * D;
    bf16_bits *l = interleaved ? h + 64 : w_lo + row * D;
    for (int q = threadIdx.x; q < D; q += 256) {
        const int at = interleaved ? q + (q & ~63) : q;   // 128 (q / 64) + q % 64
        if (d >= D) {
            h[at] = l[at] = 0;
            continue;
        }
        const double y = ident ? (q == d ? 1.0 : 0.0)
                               : Y_all[static_cast<size_t>(blk) * D * Qp + static_cast<size_t>(d) * Qp + q];
        const bf16_bits hb = f32_to_bf16_rne(static_cast<float>(y));
        h[at] = hb;
        l[at] = f32_to_bf16_rne(static_cast<float>(y - static_cast<double>(bf16_to_f32(hb))));
    }
}

template <typename TIn, typename TOut>
__global__ __launch_bounds__(256) void k_copy_rows(const TIn *src, int64_t ld_in, int cols,
                                                   TOut *dst, int64_t ld_out) {
    const int r = blockIdx.y;
    for (int c = blockIdx.x * 256 + threadIdx.x; c < cols; c += gridDim.x * 256)
        store_out_d<TOut>(dst + static_cast<int64_t>(r) * ld_out + c, load_in_d<TIn>(src + static_cast<int64_t>(r) * ld_in + c));
}

template <typename TIn, typename TOut>
hipError_t launch_solve(const WsLayout &w, int D, int n_blocks, const void *g, int64_t ld_in, int Q,
                        void *out, int64_t ld_out, hipStream_t s) {
    hipLaunchKernelGGL(k_diag_inv, dim3(tiles_of(D), n_blocks), dim3(64), 0, s, w.A, D, w.Linv);
    const dim3 grid(static_cast<unsigned>(padded_q(Q) / NB), static_cast<unsigned>(n_blocks));
    hipLaunchKernelGGL((k_trsm_f64<TIn, TOut>), grid, dim3(256), 0, s, w.A, w.Linv, D, static_cast<const TIn *>(g),
                       ld_in, Q, padded_q(Q), w.Y, w.Z, static_cast<TOut *>(out), ld_out);
    return hipGetLastError();
}

}  // namespace

inline size_t w_half_bytes(int D, int n_blocks) {
    const size_t Dp = static_cast<size_t>(D + 255) / 256 * 256;
    return align256(sizeof(bf16_bits) * static_cast<size_t>(n_blocks) * Dp * D);
}

size_t self_influence_ws_bytes(int D, int n_blocks) {
    return precond_ws_bytes(D, n_blocks, D) + 2 * w_half_bytes(D, n_blocks);
}

bf16_bits *self_influence_w(void *ws, int D, int n_blocks, bool lo) {
    char *p = static_cast<char *>(ws) + precond_ws_bytes(D, n_blocks, D);
    if (lo) p += w_half_bytes(D, n_blocks);
    return reinterpret_cast<bf16_bits *>(p);
}

size_t precond_ws_bytes(int D, int n_blocks, int Q) {
    const size_t nb = static_cast<size_t>(n_blocks);
    return align256(sizeof(double) * nb * D * D) + align256(sizeof(double) * nb) + align256(sizeof(int) * nb) +
           align256(sizeof(double) * nb * tiles_of(D) * NB * NB) +
           2 * align256(sizeof(double) * nb * D * padded_q(Q));
}

int *precond_info_ptr(void *ws, int D, int n_blocks) { return ws_layout(ws, D, n_blocks, 0).info; }

namespace {
// Dispatch over the element types of an input and an output (dtype codes).
template <typename F>
hipError_t with_types(int in_dt, int out_dt, F &&f) {
    auto out = [&](auto in_tag) -> hipError_t {
        using TI = decltype(in_tag);
        if (out_dt == kBF16) return f(TI{}, bf16_bits{});
        if (out_dt == kF64) return f(TI{}, double{});
        return f(TI{}, float{});
    };
    if (in_dt == kBF16) return out(bf16_bits{});
    if (in_dt == kF64) return out(double{});
    return out(float{});
}
}  // namespace

hipError_t launch_copy_rows(const void *src, int in_dt, int64_t ld_in, int rows, int cols,
                            void *dst, int out_dt, int64_t ld_out, hipStream_t s) {
    if (rows == 0 || cols == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(min((cols + 255) / 256, 64)), static_cast<unsigned>(rows));
    return with_types(in_dt, out_dt, [&](auto ti, auto to) {
        using TI = decltype(ti);
        using TO = decltype(to);
        hipLaunchKernelGGL((k_copy_rows<TI, TO>), grid, dim3(256), 0, s, static_cast<const TI *>(src), ld_in,
                           cols, static_cast<TO *>(dst), ld_out);
        return hipGetLastError();
    });
}

hipError_t launch_precondition(const void *S, bool s_f64, int D, int n_blocks, int64_t N, double damp_ratio,
                               const void *g_test, int in_dt, int64_t ld_in, int Q, void *g_out, int out_dt,
                               int64_t ld_out, void *ws, hipStream_t s) {
    const WsLayout w = ws_layout(ws, D, n_blocks, Q);
    if (s_f64) {
        const double *Sd = static_cast<const double *>(S);
        hipLaunchKernelGGL(k_lambda<double>, dim3(n_blocks), dim3(256), 0, s, Sd, D, N, damp_ratio, w.lam);
        hipLaunchKernelGGL(k_form<double>, dim3(D, n_blocks), dim3(256), 0, s, Sd, D, N, w.lam, w.A, w.info);
    } else {
        const float *Sf = static_cast<const float *>(S);
        hipLaunchKernelGGL(k_lambda<float>, dim3(n_blocks), dim3(256), 0, s, Sf, D, N, damp_ratio, w.lam);
        hipLaunchKernelGGL(k_form<float>, dim3(D, n_blocks), dim3(256), 0, s, Sf, D, N, w.lam, w.A, w.info);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    for (int k0 = 0; k0 < D; k0 += NB) {
        hipLaunchKernelGGL(k_potrf_diag, dim3(n_blocks), dim3(64), 0, s, w.A, D, k0, w.info);
        const int rest = D - k0 - NB;
        if (rest > 0) {
            const int nt = (rest + NB - 1) / NB;
            hipLaunchKernelGGL(k_trsm_panel, dim3(nt, n_blocks), dim3(64), 0, s, w.A, D, k0);
            hipLaunchKernelGGL(k_syrk_update, dim3(nt * (nt + 1) / 2, n_blocks), dim3(256), 0, s, w.A, D, k0, nt);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (Q == 0) return hipSuccess;
    return with_types(in_dt, out_dt, [&](auto ti, auto to) {
        return launch_solve<decltype(ti), decltype(to)>(w, D, n_blocks, g_test, ld_in, Q, g_out, ld_out, s);
    });
}

hipError_t launch_inverse_factor(const float *S, int D, int n_blocks, int64_t N, double damp_ratio,
                                 bool interleaved, void *ws, hipStream_t s) {
    const WsLayout w = ws_layout(ws, D, n_blocks, D);
    bf16_bits *hi = self_influence_w(ws, D, n_blocks, false), *lo = self_influence_w(ws, D, n_blocks, true);
    const bool ident = damp_ratio < 0;
    if (!ident) {
        // factor (status words as for the preconditioner), then L^{-1} = forward solve of I
        const hipError_t e = launch_precondition(S, false, D, n_blocks, N, damp_ratio, nullptr, kF32, D, 0,
                                                 nullptr, kF32, D, ws, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_diag_inv, dim3(tiles_of(D), n_blocks), dim3(64), 0, s, w.A, D, w.Linv);
        const dim3 grid(static_cast<unsigned>(padded_q(D) / NB), static_cast<unsigned>(n_blocks));
        hipLaunchKernelGGL((k_trsm_f64<float, float, true>), grid, dim3(256), 0, s, w.A, w.Linv, D,
                           static_cast<const float *>(nullptr), int64_t{0}, D, padded_q(D), w.Y, w.Z,
                           static_cast<float *>(nullptr), int64_t{0});
    } else {
        hipLaunchKernelGGL(k_clear_info, dim3(1), dim3(256), 0, s, w.info, n_blocks);
    }
    hipLaunchKernelGGL(k_split_w, dim3((D + 255) / 256 * 256, n_blocks), dim3(256), 0, s, w.Y, D, padded_q(D),
                       ident, interleaved, hi, lo);
    return hipGetLastError();
}

}  // namespace logra
