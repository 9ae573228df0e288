// Damped inverse applied to test gradients, per layer block (the iHVP step of
// the influence function, Sec. 2 Eq. (2), in the projected space of Eq. (3)):
//
//   C = S / N,  lambda = r * tr(C) / D   (r x mean eigenvalue, App. C)
//   out_q = (C + lambda I)^{-1} g_q
//
// All arithmetic is float64.  Steps, each batched over layer blocks
// (blockIdx.y):
//   1. lambda per block (fixed-order tree sum of the diagonal);
//   2. A = S/N + lambda I into the workspace (lower triangle);
//   3. blocked right-looking Cholesky, 64-wide panels: factor the diagonal
//      block in LDS, solve the panel below it, SYRK-update the trailing
//      matrix;  a non-positive pivot sets the block's status word;
//   4. forward and backward substitution for up to 16 right-hand sides per
//      workgroup, the right-hand sides resident in LDS, L streamed through
//      LDS in coalesced 64x64 tiles, the 64x64 triangles solved one row at a
//      time with a fixed-order wavefront reduction.
#include "common.h"
#include "internal.h"

namespace logra {
namespace {

constexpr int NB = 64;   // panel width / tile edge
constexpr int LT = NB + 1;

struct WsLayout {
    double *A;
    double *lam;
    int *info;
};

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

inline WsLayout ws_layout(void *ws, int D, int n_blocks) {
    char *p = static_cast<char *>(ws);
    WsLayout w;
    w.A = reinterpret_cast<double *>(p);
    p += align256(sizeof(double) * static_cast<size_t>(n_blocks) * D * D);
    w.lam = reinterpret_cast<double *>(p);
    p += align256(sizeof(double) * n_blocks);
    w.info = reinterpret_cast<int *>(p);
    return w;
}

__global__ __launch_bounds__(256) void k_lambda(const float *S, int D, int64_t N, double r,
                                                double *lam) {
    __shared__ double part[256];
    const int blk = blockIdx.x;
    const float *Sb = S + static_cast<size_t>(blk) * D * D;
    double s = 0.0;
    for (int d = threadIdx.x; d < D; d += 256) s += static_cast<double>(Sb[static_cast<size_t>(d) * D + d]);
    part[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) lam[blk] = r * (part[0] / static_cast<double>(N)) / static_cast<double>(D);
}

__global__ __launch_bounds__(256) void k_form(const float *S, int D, int64_t N, const double *lam,
                                              double *A, int *info) {
    const int blk = blockIdx.y, i = blockIdx.x;
    const float *Sr = S + (static_cast<size_t>(blk) * D + i) * D;
    double *Ar = A + (static_cast<size_t>(blk) * D + i) * D;
    const double inv = 1.0 / static_cast<double>(N);
    for (int j = threadIdx.x; j <= i; j += 256) {
        double v = static_cast<double>(Sr[j]) * inv;
        if (j == i) v += lam[blk];
        Ar[j] = v;
    }
    if (i == 0 && threadIdx.x == 0) info[blk] = 0;
}

// Unblocked Cholesky of the nb x nb diagonal block at (k0, k0); one wave.
__global__ __launch_bounds__(64) void k_potrf_diag(double *A_all, int D, int k0, int *info) {
    __shared__ double a[NB * LT];
    const int blk = blockIdx.x, t = threadIdx.x;
    double *A = A_all + static_cast<size_t>(blk) * D * D;
    const int nb = min(NB, D - k0);
    for (int i = 0; i < nb; ++i)
        if (t <= i) a[i * LT + t] = A[static_cast<size_t>(k0 + i) * D + k0 + t];
    __syncthreads();
    for (int j = 0; j < nb; ++j) {
        if (t == 0) {
            double piv = a[j * LT + j];
            if (!(piv > 0.0)) {
                if (info[blk] == 0) info[blk] = k0 + j + 1;
                piv = 1.0;   // keep going; the result is reported as not PD
            }
            a[j * LT + j] = sqrt(piv);
        }
        __syncthreads();
        if (t > j && t < nb) a[t * LT + j] /= a[j * LT + j];
        __syncthreads();
        if (t > j && t < nb) {
            const double lij = a[t * LT + j];
            for (int k = j + 1; k <= t; ++k) a[t * LT + k] -= lij * a[k * LT + j];
        }
        __syncthreads();
    }
    for (int i = 0; i < nb; ++i)
        if (t <= i) A[static_cast<size_t>(k0 + i) * D + k0 + t] = a[i * LT + t];
}

// Rows below the diagonal block: L21 = A21 L11^{-T}; one row per thread.
__global__ __launch_bounds__(64) void k_trsm_panel(double *A_all, int D, int k0) {
    __shared__ double l11[NB * LT];
    __shared__ double x[NB * LT];
    const int blk = blockIdx.y, t = threadIdx.x;
    double *A = A_all + static_cast<size_t>(blk) * D * D;
    const int nb = min(NB, D - k0);
    const int r0 = k0 + nb + blockIdx.x * NB;
    const int nr = min(NB, D - r0);
    for (int i = 0; i < nb; ++i) l11[i * LT + t] = (t <= i && t < nb) ? A[static_cast<size_t>(k0 + i) * D + k0 + t] : 0.0;
    for (int i = 0; i < nr; ++i) x[i * LT + t] = (t < nb) ? A[static_cast<size_t>(r0 + i) * D + k0 + t] : 0.0;
    __syncthreads();
    if (t < nr) {
        double *xr = x + t * LT;
        for (int j = 0; j < nb; ++j) {
            double s = xr[j];
            for (int m = 0; m < j; ++m) s -= xr[m] * l11[j * LT + m];
            xr[j] = s / l11[j * LT + j];
        }
    }
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

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Forward (L y = g) and backward (L^T z = y) substitution for R right-hand
// sides of one block; y lives in LDS as y[d * R + r].
template <typename TIn, typename TOut>
__global__ __launch_bounds__(256) void k_solve(const double *A_all, int D, int R, const TIn *g,
                                               int64_t ld_in, int Q, TOut *out, int64_t ld_out) {
    extern __shared__ double smem[];
    double *Lt = smem;              // [NB][LT]
    double *y = smem + NB * LT;     // [D][R]
    const int blk = blockIdx.y, q0 = blockIdx.x * R;
    const double *L = A_all + static_cast<size_t>(blk) * D * D;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nq = min(R, Q - q0);

    for (int r = 0; r < R; ++r)
        for (int d = tid; d < D; d += 256)
            y[d * R + r] = (r < nq) ? load_in_d<TIn>(g + static_cast<int64_t>(q0 + r) * ld_in + static_cast<int64_t>(blk) * D + d) : 0.0;
    __syncthreads();

    const int nblk = (D + NB - 1) / NB;
    // ---------------- forward ----------------
    for (int bi = 0; bi < nblk; ++bi) {
        const int i0 = bi * NB, nbi = min(NB, D - i0);
        double acc[4] = {0.0, 0.0, 0.0, 0.0};
        for (int m0 = 0; m0 < i0; m0 += NB) {
            for (int e = tid; e < NB * NB; e += 256) {
                const int r = e / NB, c = e - (e / NB) * NB;
                Lt[r * LT + c] = (r < nbi) ? L[static_cast<size_t>(i0 + r) * D + m0 + c] : 0.0;
            }
            __syncthreads();
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int p = tid + 256 * u;
                const int i = p & 63, r = p >> 6;
                if (r < R) {
                    double s = acc[u];
                    for (int m = 0; m < NB; ++m) s = fma(Lt[i * LT + m], y[(m0 + m) * R + r], s);
                    acc[u] = s;
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int p = tid + 256 * u;
            const int i = p & 63, r = p >> 6;
            if (r < R && i < nbi) y[(i0 + i) * R + r] -= acc[u];
        }
        for (int e = tid; e < NB * NB; e += 256) {
            const int r = e / NB, c = e - (e / NB) * NB;
            Lt[r * LT + c] = (r < nbi && c <= r) ? L[static_cast<size_t>(i0 + r) * D + i0 + c] : 0.0;
        }
        __syncthreads();
        for (int r = wave; r < R; r += 4) {
            double ym = (lane < nbi) ? y[(i0 + lane) * R + r] : 0.0;
            for (int i = 0; i < nbi; ++i) {
                const double s = wave_sum(lane < i ? Lt[i * LT + lane] * ym : 0.0);
                if (lane == i) ym = (ym - s) / Lt[i * LT + i];
            }
            if (lane < nbi) y[(i0 + lane) * R + r] = ym;
        }
        __syncthreads();
    }
    // ---------------- backward ----------------
    for (int bi = nblk - 1; bi >= 0; --bi) {
        const int i0 = bi * NB, nbi = min(NB, D - i0);
        double acc[4] = {0.0, 0.0, 0.0, 0.0};
        for (int m0 = i0 + NB; m0 < D; m0 += NB) {
            const int nm = min(NB, D - m0);
            for (int e = tid; e < NB * NB; e += 256) {
                const int r = e / NB, c = e - (e / NB) * NB;   // r: row m, c: column i
                Lt[r * LT + c] = (r < nm && c < nbi) ? L[static_cast<size_t>(m0 + r) * D + i0 + c] : 0.0;
            }
            __syncthreads();
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int p = tid + 256 * u;
                const int i = p & 63, r = p >> 6;
                if (r < R) {
                    double s = acc[u];
                    for (int m = 0; m < nm; ++m) s = fma(Lt[m * LT + i], y[(m0 + m) * R + r], s);
                    acc[u] = s;
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int p = tid + 256 * u;
            const int i = p & 63, r = p >> 6;
            if (r < R && i < nbi) y[(i0 + i) * R + r] -= acc[u];
        }
        for (int e = tid; e < NB * NB; e += 256) {
            const int r = e / NB, c = e - (e / NB) * NB;
            Lt[r * LT + c] = (r < nbi && c <= r) ? L[static_cast<size_t>(i0 + r) * D + i0 + c] : 0.0;
        }
        __syncthreads();
        for (int r = wave; r < R; r += 4) {
            double zm = (lane < nbi) ? y[(i0 + lane) * R + r] : 0.0;
            for (int i = nbi - 1; i >= 0; --i) {
                const double s = wave_sum((lane > i && lane < nbi) ? Lt[lane * LT + i] * zm : 0.0);
                if (lane == i) zm = (zm - s) / Lt[i * LT + i];
            }
            if (lane < nbi) y[(i0 + lane) * R + r] = zm;
        }
        __syncthreads();
    }
    for (int r = 0; r < nq; ++r)
        for (int d = tid; d < D; d += 256)
            store_out_d<TOut>(out + static_cast<int64_t>(q0 + r) * ld_out + static_cast<int64_t>(blk) * D + d, y[d * R + r]);
}

template <typename TIn, typename TOut>
__global__ __launch_bounds__(256) void k_copy_rows(const TIn *src, int64_t ld_in, int cols,
                                                   TOut *dst, int64_t ld_out) {
    const int r = blockIdx.y;
    for (int c = blockIdx.x * 256 + threadIdx.x; c < cols; c += gridDim.x * 256)
        store_out_d<TOut>(dst + static_cast<int64_t>(r) * ld_out + c, load_in_d<TIn>(src + static_cast<int64_t>(r) * ld_in + c));
}

inline int rhs_per_group(int D) {
    int R = 12288 / D;
    if (R > 16) R = 16;
    if (R < 1) R = 1;
    return R;
}

template <typename TIn, typename TOut>
hipError_t launch_solve(const double *A, int D, int n_blocks, const void *g, int64_t ld_in, int Q,
                        void *out, int64_t ld_out, hipStream_t s) {
    const int R = rhs_per_group(D);
    const size_t smem = sizeof(double) * (static_cast<size_t>(NB) * LT + static_cast<size_t>(D) * R);
    const auto kern = k_solve<TIn, TOut>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(smem));
    if (e != hipSuccess) return e;
    const dim3 grid(static_cast<unsigned>((Q + R - 1) / R), static_cast<unsigned>(n_blocks));
    hipLaunchKernelGGL(kern, grid, dim3(256), smem, s, A, D, R, static_cast<const TIn *>(g), ld_in, Q,
                       static_cast<TOut *>(out), ld_out);
    return hipGetLastError();
}

}  // namespace

size_t precond_ws_bytes(int D, int n_blocks, int /*Q*/) {
    return align256(sizeof(double) * static_cast<size_t>(n_blocks) * D * D) +
           align256(sizeof(double) * n_blocks) + align256(sizeof(int) * n_blocks);
}

int *precond_info_ptr(void *ws, int D, int n_blocks) { return ws_layout(ws, D, n_blocks).info; }

hipError_t launch_copy_rows(const void *src, bool bf16_in, int64_t ld_in, int rows, int cols,
                            void *dst, bool bf16_out, int64_t ld_out, hipStream_t s) {
    if (rows == 0 || cols == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(min((cols + 255) / 256, 64)), static_cast<unsigned>(rows));
    if (bf16_in && bf16_out)
        hipLaunchKernelGGL((k_copy_rows<bf16_bits, bf16_bits>), grid, dim3(256), 0, s, static_cast<const bf16_bits *>(src), ld_in, cols, static_cast<bf16_bits *>(dst), ld_out);
    else if (bf16_in)
        hipLaunchKernelGGL((k_copy_rows<bf16_bits, float>), grid, dim3(256), 0, s, static_cast<const bf16_bits *>(src), ld_in, cols, static_cast<float *>(dst), ld_out);
    else if (bf16_out)
        hipLaunchKernelGGL((k_copy_rows<float, bf16_bits>), grid, dim3(256), 0, s, static_cast<const float *>(src), ld_in, cols, static_cast<bf16_bits *>(dst), ld_out);
    else
        hipLaunchKernelGGL((k_copy_rows<float, float>), grid, dim3(256), 0, s, static_cast<const float *>(src), ld_in, cols, static_cast<float *>(dst), ld_out);
    return hipGetLastError();
}

hipError_t launch_precondition(const float *S, int D, int n_blocks, int64_t N, double damp_ratio,
                               const void *g_test, bool bf16_in, int64_t ld_in, int Q, void *g_out,
                               bool bf16_out, int64_t ld_out, void *ws, hipStream_t s) {
    const WsLayout w = ws_layout(ws, D, n_blocks);
    hipLaunchKernelGGL(k_lambda, dim3(n_blocks), dim3(256), 0, s, S, D, N, damp_ratio, w.lam);
    hipLaunchKernelGGL(k_form, dim3(D, n_blocks), dim3(256), 0, s, S, D, N, w.lam, w.A, w.info);
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
    if (bf16_in && bf16_out) return launch_solve<bf16_bits, bf16_bits>(w.A, D, n_blocks, g_test, ld_in, Q, g_out, ld_out, s);
    if (bf16_in) return launch_solve<bf16_bits, float>(w.A, D, n_blocks, g_test, ld_in, Q, g_out, ld_out, s);
    if (bf16_out) return launch_solve<float, bf16_bits>(w.A, D, n_blocks, g_test, ld_in, Q, g_out, ld_out, s);
    return launch_solve<float, float>(w.A, D, n_blocks, g_test, ld_in, Q, g_out, ld_out, s);
}

}  // namespace logra
