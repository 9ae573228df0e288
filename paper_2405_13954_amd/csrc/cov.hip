// Projected Fisher covariance (Sec. 2 Eq. (3); App. D Assumption 1):
//
//   S_l += sum_b g_b,l g_b,l^T      for each column block l of width D
//
// One workgroup per upper-triangle 64x64 tile (I <= J) of one block.  The
// contraction runs over examples b in chunks of 32: the g rows of the chunk
// are read with 128-bit coalesced loads and written transposed into LDS
// ([column][example]), from where each lane reads its 8 consecutive examples
// as one MFMA operand (16x16x32 bf16, fp32 accumulation).  fp32 inputs use a
// plain fp32 FMA loop.  The fp64 form (S in float64, for fp32 or fp64 rows)
// forms every product and sum in float64: a product of two fp32 values is
// exact there.  The tile is then added to S (coalesced
// read-modify-write of the upper tile) and written mirrored to the lower
// tile through LDS, so S stays exactly symmetric.
#include "common.h"
#include "internal.h"

namespace logra {
namespace {

constexpr int CT = 64;   // tile edge
constexpr int BK = 32;   // examples per contraction chunk (bf16 MFMA K)

__device__ __forceinline__ void tile_coords(int t, int nt, int &ti, int &tj) {
    // t enumerates the upper triangle row by row: (0,0),(0,1)..(0,nt-1),(1,1),...
    int i = 0;
    while (t >= nt - i) {
        t -= nt - i;
        ++i;
    }
    ti = i;
    tj = i + t;
}

// Add the computed 64x64 tile c (LDS, row-major with stride CT+1) into S and
// mirror it.  Diagonal tiles only use entries r <= c of the upper triangle.
// Off-diagonal tiles of an S whose rows are 16-byte aligned and whose edge is
// a multiple of 64 take the vector form: thread t owns row t / 4 of the tile
// and its 16 columns 16 (t % 4) .. +15, loads them as four 128-bit loads all
// in flight at once, adds, stores, and writes the mirrored tile the same way
// (row t / 4 of the transposed tile, gathered from LDS).
template <typename TS>
__device__ __forceinline__ void add_and_mirror(TS *S, int D, int I, int J, TS *ct, bool diag) {
    const int tid = threadIdx.x;
    if constexpr (sizeof(TS) == 4) {
        if (!diag && D % CT == 0 && (reinterpret_cast<uintptr_t>(S) & 15) == 0) {
            const int r = tid >> 2, c0 = 16 * (tid & 3);
            f32x4 *row = reinterpret_cast<f32x4 *>(S + static_cast<size_t>(I + r) * D + J + c0);
            f32x4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = row[u];
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    v[u][e] += ct[r * (CT + 1) + c0 + 4 * u + e];
                    ct[r * (CT + 1) + c0 + 4 * u + e] = v[u][e];
                }
#pragma unroll
            for (int u = 0; u < 4; ++u) row[u] = v[u];
            __syncthreads();
            // mirrored: S[J + c][I + i] = tile[i][c], thread t writes c = t / 4, i = 16 (t % 4) .. +15
            f32x4 *mrow = reinterpret_cast<f32x4 *>(S + static_cast<size_t>(J + r) * D + I + c0);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                f32x4 m;
#pragma unroll
                for (int e = 0; e < 4; ++e) m[e] = ct[(c0 + 4 * u + e) * (CT + 1) + r];
                mrow[u] = m;
            }
            return;
        }
    }
    for (int e = tid; e < CT * CT; e += blockDim.x) {
        const int r = e / CT, c = e - (e / CT) * CT;
        const int i = I + r, j = J + c;
        if (i < D && j < D && (!diag || r <= c)) {
            TS *p = S + static_cast<size_t>(i) * D + j;
            const TS v = *p + ct[r * (CT + 1) + c];
            *p = v;
            ct[r * (CT + 1) + c] = v;
        }
    }
    __syncthreads();
    for (int e = tid; e < CT * CT; e += blockDim.x) {
        const int c = e / CT, r = e - (e / CT) * CT;   // consecutive threads: consecutive r
        const int i = I + r, j = J + c;
        if (i < D && j < D && (diag ? r < c : true)) S[static_cast<size_t>(j) * D + i] = ct[r * (CT + 1) + c];
    }
}

__global__ __launch_bounds__(256) void k_cov_bf16(const bf16_bits *g, int64_t ld, int B, int D,
                                                  int nt, float *S_all) {
    __shared__ __attribute__((aligned(16))) bf16_bits gi[CT][BK + 8];  // [column][example]
    __shared__ __attribute__((aligned(16))) bf16_bits gj[CT][BK + 8];
    __shared__ float ct[CT * (CT + 1)];

    const int blk = blockIdx.y;
    int ti, tj;
    tile_coords(blockIdx.x, nt, ti, tj);
    const int I = ti * CT, J = tj * CT;
    const bool diag = ti == tj;
    const bf16_bits *gb = g + static_cast<size_t>(blk) * D;
    float *S = S_all + static_cast<size_t>(blk) * D * D;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row = lane & 15, kg = lane >> 4;
    f32x4 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // staging: thread -> (example r = tid / 8, 8 columns c8 = 8 * (tid % 8))
    const int sr = tid >> 3, sc = (tid & 7) * 8;
    for (int b0 = 0; b0 < B; b0 += BK) {
        const int b = b0 + sr;
        u32x4 vi = {0u, 0u, 0u, 0u}, vj = {0u, 0u, 0u, 0u};
        if (b < B) {
            const bf16_bits *rowp = gb + static_cast<int64_t>(b) * ld;
            if (I + sc < D) vi = ld128(rowp + I + sc);
            if (!diag && J + sc < D) vj = ld128(rowp + J + sc);
        }
        __syncthreads();  // previous chunk's operands fully consumed
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint32_t wi = vi[e >> 1], wj = vj[e >> 1];
            gi[sc + e][sr] = static_cast<bf16_bits>((e & 1) ? (wi >> 16) : (wi & 0xffffu));
            if (!diag) gj[sc + e][sr] = static_cast<bf16_bits>((e & 1) ? (wj >> 16) : (wj & 0xffffu));
        }
        __syncthreads();
        const bf16_bits(*gjs)[BK + 8] = diag ? gi : gj;
        const bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4 *>(&gi[16 * wave + row][8 * kg]));
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const bf16x8 bb = as_bf16x8(*reinterpret_cast<const u32x4 *>(&gjs[16 * j + row][8 * kg]));
            acc[j] = mfma16_bf16(a, bb, acc[j]);
        }
    }
    // result: rows 16*wave + 4*kg + r, columns 16*j + row
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) ct[(16 * wave + 4 * kg + r) * (CT + 1) + 16 * j + row] = acc[j][r];
    __syncthreads();
    add_and_mirror(S, D, I, J, ct, diag);
}

__global__ __launch_bounds__(256) void k_cov_f32(const float *g, int64_t ld, int B, int D, int nt,
                                                 float *S_all) {
    __shared__ float ct[CT * (CT + 1)];
    const int blk = blockIdx.y;
    int ti, tj;
    tile_coords(blockIdx.x, nt, ti, tj);
    const int I = ti * CT, J = tj * CT;
    const bool diag = ti == tj;
    const float *gb = g + static_cast<size_t>(blk) * D;
    float *S = S_all + static_cast<size_t>(blk) * D * D;
    for (int e = threadIdx.x; e < CT * CT; e += blockDim.x) {
        const int r = e / CT, c = e - (e / CT) * CT;
        const int i = I + r, j = J + c;
        float s = 0.f;
        if (i < D && j < D)
            for (int b = 0; b < B; ++b) {
                const float *rowp = gb + static_cast<int64_t>(b) * ld;
                s = __builtin_fmaf(rowp[i], rowp[j], s);
            }
        ct[r * (CT + 1) + c] = s;
    }
    __syncthreads();
    add_and_mirror(S, D, I, J, ct, diag);
}

// float64 statistics: rows of fp32 or fp64, every product and sum in float64.
template <typename TG>
__global__ __launch_bounds__(256) void k_cov_f64(const TG *g, int64_t ld, int B, int D, int nt,
                                                 double *S_all) {
    __shared__ double ct[CT * (CT + 1)];
    const int blk = blockIdx.y;
    int ti, tj;
    tile_coords(blockIdx.x, nt, ti, tj);
    const int I = ti * CT, J = tj * CT;
    const bool diag = ti == tj;
    const TG *gb = g + static_cast<size_t>(blk) * D;
    double *S = S_all + static_cast<size_t>(blk) * D * D;
    for (int e = threadIdx.x; e < CT * CT; e += blockDim.x) {
        const int r = e / CT, c = e - (e / CT) * CT;
        const int i = I + r, j = J + c;
        double s = 0.0;
        if (i < D && j < D)
            for (int b = 0; b < B; ++b) {
                const TG *rowp = gb + static_cast<int64_t>(b) * ld;
                s = fma(load_in_d<TG>(rowp + i), load_in_d<TG>(rowp + j), s);
            }
        ct[r * (CT + 1) + c] = s;
    }
    __syncthreads();
    add_and_mirror(S, D, I, J, ct, diag);
}

}  // namespace

hipError_t launch_cov(const void *g, bool bf16, int64_t ld, int B, int D, int n_blocks, float *S,
                      hipStream_t s) {
    if (B == 0 || n_blocks == 0) return hipSuccess;
    const int nt = (D + CT - 1) / CT;
    const dim3 grid(static_cast<unsigned>(nt * (nt + 1) / 2), static_cast<unsigned>(n_blocks));
    if (bf16)
        hipLaunchKernelGGL(k_cov_bf16, grid, dim3(256), 0, s, static_cast<const bf16_bits *>(g), ld, B,
                           D, nt, S);
    else
        hipLaunchKernelGGL(k_cov_f32, grid, dim3(256), 0, s, static_cast<const float *>(g), ld, B, D,
                           nt, S);
    return hipGetLastError();
}

hipError_t launch_cov_f64(const void *g, bool f64_rows, int64_t ld, int B, int D, int n_blocks, double *S,
                          hipStream_t s) {
    if (B == 0 || n_blocks == 0) return hipSuccess;
    const int nt = (D + CT - 1) / CT;
    const dim3 grid(static_cast<unsigned>(nt * (nt + 1) / 2), static_cast<unsigned>(n_blocks));
    if (f64_rows)
        hipLaunchKernelGGL(k_cov_f64<double>, grid, dim3(256), 0, s, static_cast<const double *>(g), ld, B, D,
                           nt, S);
    else
        hipLaunchKernelGGL(k_cov_f64<float>, grid, dim3(256), 0, s, static_cast<const float *>(g), ld, B, D,
                           nt, S);
    return hipGetLastError();
}

}  // namespace logra
