// Fused per-example structured gradient projection (LoGra, Sec. 3.1, Eq. (5)).
//
//   G_b = sum_t m_bt (P_out dy_bt)(P_in x_bt)^T        (k_out x k_in, fp32)
//
// One workgroup (4 waves) owns a 64-token tile of one example of one layer.
//  1. Projection: x'[64 x k_in] = X_tile P_in^T and dy'[64 x k_out] =
//     dY_tile P_out^T on the matrix cores (16x16x32 bf16 or 16x16x4 fp32,
//     fp32 accumulation).  The n-contraction is split into 32-wide steps
//     dealt round-robin to the waves; each lane feeds a 128-bit global load
//     straight into its MFMA operand (row = token for X, row = projection
//     dimension for P), so x and dy are read from HBM once with no LDS
//     staging.  Masked and out-of-range tokens are never loaded (their
//     operand is zero), so NaN/Inf in padding cannot leak.
//  2. The four waves' partial x'/dy' are folded in a fixed order through
//     LDS (deterministic).
//  3. The per-tile sum over tokens of dy'_t x'_t^T runs in fp32 from LDS,
//     4x4 outputs per thread.
// A second kernel adds the per-tile partials of each example in tile order
// and writes G_b (fp32 or bf16) into the caller's store row.
#include "common.h"
#include "internal.h"

namespace logra {
namespace {

constexpr int TT = kProjTile;  // tokens per tile
constexpr int NT = 256;        // threads per workgroup
constexpr int NW = NT / kWave; // waves per workgroup

struct ProjArgs {
    ProjGroup grp;
    const uint8_t *mask;
    float *partial;
    int B, T, tpe;  // tpe = tiles per example
    int k_in, k_out;
};

template <typename TIn>
struct InTraits;
template <>
struct InTraits<bf16_bits> {
    static constexpr int kElems = 8;   // elements per 128-bit lane load
    static constexpr int kStep = 32;   // contraction width of one step (4 lane groups x 8)
};
template <>
struct InTraits<float> {
    static constexpr int kElems = 4;
    static constexpr int kStep = 16;
};

template <int KT>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[4][KT], const u32x4 (&xa)[4],
                                         const u32x4 (&pb)[KT], bf16_bits) {
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int j = 0; j < KT; ++j) acc[m][j] = mfma16_bf16(as_bf16x8(xa[m]), as_bf16x8(pb[j]), acc[m][j]);
}

template <int KT>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[4][KT], const u32x4 (&xa)[4],
                                         const u32x4 (&pb)[KT], float) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int j = 0; j < KT; ++j)
                acc[m][j] = mfma16_f32(__uint_as_float(xa[m][e]), __uint_as_float(pb[j][e]), acc[m][j]);
}

// One wave's share of  A'[64 x 16KT] = A_tile[64 x n] * P^T  (P: k rows of n).
// Contraction steps s = wave, wave + NW, ... ; two register stages so that
// the next step's loads are in flight while the current step multiplies.
template <int KT, typename TIn>
__device__ __forceinline__ void project_part(f32x4 (&acc)[4][KT], const TIn *A, const TIn *P,
                                             int n, int k, const bool (&tok_ok)[4], int wave,
                                             int lane) {
    constexpr int E = InTraits<TIn>::kElems;
    constexpr int S = InTraits<TIn>::kStep;
    const int row = lane & 15;
    const int kg = lane >> 4;
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int j = 0; j < KT; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const TIn *arow[4];
    const TIn *prow[KT];
    bool p_ok[KT];
#pragma unroll
    for (int m = 0; m < 4; ++m) arow[m] = A + static_cast<size_t>(16 * m + row) * n + kg * E;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
        p_ok[j] = (16 * j + row) < k;
        prow[j] = P + static_cast<size_t>(p_ok[j] ? 16 * j + row : 0) * n + kg * E;
    }
    const int nsteps = (n + S - 1) / S;

    auto load = [&](int s, u32x4(&xa)[4], u32x4(&pb)[KT]) {
        const int off = s * S;
        const bool in_n = off + kg * E < n;
        const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int m = 0; m < 4; ++m) xa[m] = (tok_ok[m] && in_n) ? ld128_nt(arow[m] + off) : z;
#pragma unroll
        for (int j = 0; j < KT; ++j) pb[j] = (p_ok[j] && in_n) ? ld128(prow[j] + off) : z;
    };

    u32x4 xa0[4], pb0[KT], xa1[4], pb1[KT];
    int s = wave;
    if (s >= nsteps) return;
    load(s, xa0, pb0);
    while (true) {
        if (s + NW < nsteps) load(s + NW, xa1, pb1);
        mma_step<KT>(acc, xa0, pb0, TIn{});
        s += NW;
        if (s >= nsteps) break;
        if (s + NW < nsteps) load(s + NW, xa0, pb0);
        mma_step<KT>(acc, xa1, pb1, TIn{});
        s += NW;
        if (s >= nsteps) break;
    }
}

// Fold the four waves' accumulators (order ((w3 + w2) + w1) + w0) and write
// the result as dst[token][16*KT] fp32.
template <int KT>
__device__ __forceinline__ void fold_waves(f32x4 (&acc)[4][KT], f32x4 *red, float *dst, int wave,
                                           int lane) {
    f32x4 *slot = red + lane;  // red[(m*KT + j) * 64 + lane]
    if (wave == NW - 1) {
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int j = 0; j < KT; ++j) slot[(m * KT + j) * kWave] = acc[m][j];
    }
    __syncthreads();
#pragma unroll
    for (int w = NW - 2; w >= 1; --w) {
        if (wave == w) {
#pragma unroll
            for (int m = 0; m < 4; ++m)
#pragma unroll
                for (int j = 0; j < KT; ++j) slot[(m * KT + j) * kWave] = slot[(m * KT + j) * kWave] + acc[m][j];
        }
        __syncthreads();
    }
    if (wave == 0) {
        const int row = lane & 15, kg = lane >> 4;
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int j = 0; j < KT; ++j) {
                const f32x4 v = slot[(m * KT + j) * kWave] + acc[m][j];
#pragma unroll
                for (int r = 0; r < 4; ++r) dst[(16 * m + 4 * kg + r) * (16 * KT) + 16 * j + row] = v[r];
            }
    }
    __syncthreads();
}

template <int KT, typename TIn>
__global__ __launch_bounds__(NT) void k_project_tiles(ProjArgs a) {
    constexpr int KP = 16 * KT;              // padded projection width
    __shared__ float xs[TT * KP];            // x'  [token][i]
    __shared__ float ds[TT * KP];            // dy' [token][o]
    __shared__ f32x4 red[4 * KT * kWave];    // cross-wave fold slot

    const int per_layer = a.B * a.tpe;
    const int l = blockIdx.x / per_layer;
    const int rem = blockIdx.x - l * per_layer;
    const int b = rem / a.tpe;
    const int tile = rem - b * a.tpe;
    const int t0 = tile * TT;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int D = a.k_in * a.k_out;
    float *part = a.partial + (static_cast<size_t>(l * a.B + b) * a.tpe + tile) * D;

    // Token validity of the four rows this lane feeds (tokens t0 + 16m + lane%16).
    bool tok_ok[4];
    bool any = false;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const int t = t0 + 16 * m + (lane & 15);
        bool ok = t < a.T;
        if (ok && a.mask) ok = a.mask[static_cast<size_t>(b) * a.T + t] != 0;
        tok_ok[m] = ok;
        any |= ok;
    }
    if (!__syncthreads_or(any)) {  // fully masked tile: contributes zero
        for (int i = tid; i < D; i += NT) part[i] = 0.f;
        return;
    }

    const ProjLayer &L = a.grp.layer[l];
    const size_t tok0 = static_cast<size_t>(b) * a.T + t0;
    f32x4 acc[4][KT];

    project_part<KT>(acc, static_cast<const TIn *>(L.x) + tok0 * L.n_in,
                     static_cast<const TIn *>(L.p_in), L.n_in, a.k_in, tok_ok, wave, lane);
    fold_waves<KT>(acc, red, xs, wave, lane);
    project_part<KT>(acc, static_cast<const TIn *>(L.dy) + tok0 * L.n_out,
                     static_cast<const TIn *>(L.p_out), L.n_out, a.k_out, tok_ok, wave, lane);
    fold_waves<KT>(acc, red, ds, wave, lane);

    // Sum over the tile's tokens of dy'_t x'_t^T; 4x4 outputs per thread.
    constexpr int NB = 4 * KT;  // 4-wide blocks per side
    for (int blk = tid; blk < NB * NB; blk += NT) {
        const int ob = blk / NB, ib = blk - (blk / NB) * NB;
        float c[4][4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int v = 0; v < 4; ++v) c[u][v] = 0.f;
        for (int t = 0; t < TT; ++t) {
            const f32x4 dv = *reinterpret_cast<const f32x4 *>(&ds[t * KP + 4 * ob]);
            const f32x4 xv = *reinterpret_cast<const f32x4 *>(&xs[t * KP + 4 * ib]);
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v) c[u][v] = __builtin_fmaf(dv[u], xv[v], c[u][v]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int o = 4 * ob + u;
            if (o >= a.k_out) break;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int i = 4 * ib + v;
                if (i < a.k_in) part[o * a.k_in + i] = c[u][v];
            }
        }
    }
}

template <typename TOut>
__global__ __launch_bounds__(256) void k_project_reduce(ProjGroup grp, const float *partial, int B,
                                                        int tpe, int D, int64_t g_ld) {
    const int l = blockIdx.x / B;
    const int b = blockIdx.x - l * B;
    const float *p = partial + static_cast<size_t>(l * B + b) * tpe * D;
    TOut *out = static_cast<TOut *>(grp.layer[l].g_out) + static_cast<int64_t>(b) * g_ld;
    for (int i = threadIdx.x; i < D; i += blockDim.x) {
        float s = 0.f;
        for (int t = 0; t < tpe; ++t) s += p[static_cast<size_t>(t) * D + i];
        store_out<TOut>(out + i, s);
    }
}

template <int KT, typename TIn>
hipError_t launch_tiles(const ProjArgs &a, int n_layers, hipStream_t s) {
    const unsigned grid = static_cast<unsigned>(n_layers) * a.B * a.tpe;
    hipLaunchKernelGGL((k_project_tiles<KT, TIn>), dim3(grid), dim3(NT), 0, s, a);
    return hipGetLastError();
}

}  // namespace

size_t project_partial_bytes(int n_layers, int B, int T, int k_in, int k_out) {
    const size_t tpe = (static_cast<size_t>(T) + TT - 1) / TT;
    return static_cast<size_t>(n_layers) * B * tpe * k_in * k_out * sizeof(float);
}

hipError_t launch_project(const ProjGroup &grp, bool bf16_in, int B, int T, const uint8_t *mask,
                          int k_in, int k_out, bool bf16_out, int64_t g_ld, float *partial,
                          hipStream_t s) {
    if (B == 0 || T == 0 || grp.n_layers == 0) return hipSuccess;
    ProjArgs a;
    a.grp = grp;
    a.mask = mask;
    a.partial = partial;
    a.B = B;
    a.T = T;
    a.tpe = (T + TT - 1) / TT;
    a.k_in = k_in;
    a.k_out = k_out;
    const int kmax = k_in > k_out ? k_in : k_out;
    const int kt = kmax <= 16 ? 1 : kmax <= 32 ? 2 : kmax <= 64 ? 4 : 8;
    hipError_t e;
    if (bf16_in) {
        switch (kt) {
            case 1: e = launch_tiles<1, bf16_bits>(a, grp.n_layers, s); break;
            case 2: e = launch_tiles<2, bf16_bits>(a, grp.n_layers, s); break;
            case 4: e = launch_tiles<4, bf16_bits>(a, grp.n_layers, s); break;
            default: e = launch_tiles<8, bf16_bits>(a, grp.n_layers, s); break;
        }
    } else {
        switch (kt) {
            case 1: e = launch_tiles<1, float>(a, grp.n_layers, s); break;
            case 2: e = launch_tiles<2, float>(a, grp.n_layers, s); break;
            case 4: e = launch_tiles<4, float>(a, grp.n_layers, s); break;
            default: e = launch_tiles<8, float>(a, grp.n_layers, s); break;
        }
    }
    if (e != hipSuccess) return e;
    const unsigned grid = static_cast<unsigned>(grp.n_layers) * B;
    if (bf16_out)
        hipLaunchKernelGGL((k_project_reduce<bf16_bits>), dim3(grid), dim3(256), 0, s, grp, partial,
                           B, a.tpe, k_in * k_out, g_ld);
    else
        hipLaunchKernelGGL((k_project_reduce<float>), dim3(grid), dim3(256), 0, s, grp, partial, B,
                           a.tpe, k_in * k_out, g_ld);
    return hipGetLastError();
}

}  // namespace logra
