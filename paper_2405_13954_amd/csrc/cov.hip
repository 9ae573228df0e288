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
__device__ __forceinline__ void add_and_mirror(TS *S, int D, int I, int J, TS *ct, bool diag, bool lower) {
    const int tid = threadIdx.x;
    if (lower) {
        // lower triangle only: tile entry (r, c) of the upper tile (I, J) is S(J + c, I + r)
        for (int e = tid; e < CT * CT; e += blockDim.x) {
            const int c = e / CT, r = e - (e / CT) * CT;   // consecutive threads: consecutive r
            const int i = I + r, j = J + c;
            if (i < D && j < D && (!diag || r <= c)) S[static_cast<size_t>(j) * D + i] += ct[r * (CT + 1) + c];
        }
        return;
    }
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
                                                  int nt, float *S_all, bool lower) {
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
    add_and_mirror(S, D, I, J, ct, diag, lower);
}

// Strict upper triangle, row by row: (0,1),(0,2)..(0,nt-1),(1,2),...
__device__ __forceinline__ void strict_upper_coords(int t, int nt, int &ti, int &tj) {
    int i = 0;
    while (t >= nt - 1 - i) {
        t -= nt - 1 - i;
        ++i;
    }
    ti = i;
    tj = i + 1 + t;
}

// One example chunk of a wave's operands: lane (row, kg) holds examples
// b0 + 8 kg + m, m < 8, of the four features c0 + 4 row .. +3 (8 bytes each),
// read through a buffer resource so that rows at or past B read as zeros.
struct CovRows {
    uint32_t w[8][2];
};
__device__ __forceinline__ void cov_load_rows(CovRows &r, __amdgpu_buffer_rsrc_t rs, uint32_t voff,
                                              uint32_t row_bytes) {
#pragma unroll
    for (int m = 0; m < 8; ++m) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, static_cast<int>(voff + m * row_bytes), 0, 0);
        r.w[m][0] = v[0];
        r.w[m][1] = v[1];
    }
}
// MFMA operand of feature c0 + 4 row + e: element m = example 8 kg + m.
__device__ __forceinline__ bf16x8 cov_operand(const CovRows &r, int e) {
    u32x4 v;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t lo = r.w[2 * p][e >> 1], hi = r.w[2 * p + 1][e >> 1];
        v[p] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    return as_bf16x8(v);
}

// Orders one wave's LDS writes before its later reads (and reads before later
// writes): the wave's LDS operations execute in issue order, so only the
// compiler has to be kept from moving them across.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// 128-bit store at a byte offset from a wave-uniform base (a global store with
// a scalar base).  Not a buffer store: the compiler puts no wait states between
// a buffer store with a register scalar offset and the next writes of its data
// registers, and such stores were seen, under load, to write the later values.
__device__ __forceinline__ void st_f32x4(float *base, uint32_t byte_off, f32x4 v) {
    *reinterpret_cast<f32x4 *>(reinterpret_cast<char *>(base) + byte_off) = v;
}

// bf16 rows, D a multiple of 64: one wave per 64x64 tile, everything in
// registers.  The wave's 16x16x32 MFMA row index ra stands for feature
// I + 4 ra + e and its column index rb for J + 4 rb + f, so the 16 products
// (e, f) cover the tile, and lane (row, kg) holds for each (r, e) the four
// consecutive columns J + 4 row .. +3 of tile row I + 16 kg + 4 r + e.  The
// accumulators start from those S entries (128-bit reads, four whole
// 256-byte tile rows per instruction, issued with the first rows of g so the
// latencies overlap), so the products are summed onto S, and the result is
// stored back the same way (global stores).  The mirrored values of a fixed f are
// four consecutive columns of row J + 4 row + f; they are regrouped through
// LDS so that the mirror is stored in whole rows too.  Row offsets that are the same
// for the whole wave travel in the scalar offset of the buffer loads.
// Off-diagonal tiles (kDiag false) write the upper tile and its mirror;
// diagonal tiles (kDiag true, two waves per workgroup) go through the wave's
// LDS so that every entry below the diagonal is the bit copy of its upper twin.
// With kLower only the lower triangle is read and written: the tile below the
// diagonal is computed in place of the upper one and nothing is mirrored.
template <bool kDiag, bool kLower>
__global__ __launch_bounds__(256, 3) void k_cov_bf16_reg(const bf16_bits *g, int64_t ld, int B, int D, int nt,
                                                      int n_tiles, float *S_all) {
    constexpr int kWaves = kDiag && !kLower ? 2 : 4;   // waves (tiles) per workgroup
    constexpr int kHalf = 32 * (CT + 4);                // half a mirrored tile: 32 rows of 68 floats
    constexpr int kLds = kLower ? 1 : kDiag ? kWaves * CT * (CT + 1) : kWaves * kHalf;
    __shared__ __attribute__((aligned(16))) float tl[kLds];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int t = __builtin_amdgcn_readfirstlane(static_cast<int>(blockIdx.x) * kWaves + wave);
    const bool live = t < n_tiles;   // wave-uniform; every wave still reaches the barrier
    int ti = 0, tj = 0;
    if (live) {
        if (kDiag) ti = tj = t;
        else strict_upper_coords(t, nt, ti, tj);
    }
    // the lower triangle alone: the tile below the diagonal, (tj, ti)
    const int I = (kLower ? tj : ti) * CT, J = (kLower ? ti : tj) * CT;
    const int row = lane & 15, kg = lane >> 4;
    const int blk = blockIdx.y;
    const auto gs = buf_rsrc(g + static_cast<size_t>(blk) * D,
                             static_cast<uint32_t>((static_cast<int64_t>(B - 1) * ld + D) * 2));
    float *Sb = S_all + static_cast<size_t>(blk) * D * D;
    const auto ss = buf_rsrc(Sb, static_cast<uint32_t>(D) * D * 4u);
    const uint32_t row_bytes = static_cast<uint32_t>(ld) * 2u;
    // lane parts of the offsets: upper tile element (16 kg, 4 row); mirrored row
    // 4 (lane / 32) + (lane / 16) % 2 of a group of eight, piece lane % 16
    const uint32_t vu = (static_cast<uint32_t>(16 * kg) * D + 4 * row) * 4u;
    const uint32_t vm = ((4 * (lane >> 5) + ((lane >> 4) & 1)) * static_cast<uint32_t>(D) + 4 * (lane & 15)) * 4u;

    f32x4 acc[4][4];   // [e][f], element r: S(I + 16 kg + 4 r + e, J + 4 row + f)
    if (live) {
        const uint32_t va = (static_cast<uint32_t>(8 * kg) * row_bytes) + (I + 4 * row) * 2u;
        const uint32_t vb = (static_cast<uint32_t>(8 * kg) * row_bytes) + (J + 4 * row) * 2u;
        CovRows ra, rb;
        cov_load_rows(ra, gs, va, row_bytes);
        if (!kDiag) cov_load_rows(rb, gs, vb, row_bytes);
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const f32x4 v = as_f32x4(__builtin_amdgcn_raw_buffer_load_b128(
                    ss, static_cast<int>(vu), static_cast<int>(((I + 4 * r + e) * static_cast<uint32_t>(D) + J) * 4u),
                    0));
#pragma unroll
                for (int f = 0; f < 4; ++f) acc[e][f][r] = v[f];
            }
        for (int b0 = 0; b0 < B; b0 += 32) {
            if (b0 > 0) {
                cov_load_rows(ra, gs, va + static_cast<uint32_t>(b0) * row_bytes, row_bytes);
                if (!kDiag) cov_load_rows(rb, gs, vb + static_cast<uint32_t>(b0) * row_bytes, row_bytes);
            }
            bf16x8 bo[4];
#pragma unroll
            for (int f = 0; f < 4; ++f) bo[f] = cov_operand(kDiag ? ra : rb, f);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bf16x8 a = cov_operand(ra, e);
#pragma unroll
                for (int f = 0; f < 4; ++f) acc[e][f] = mfma16_bf16(a, bo[f], acc[e][f]);
            }
        }
    }
    if constexpr (kLower) {
        // the tile itself; on the diagonal only entries (i, c) with c <= i
        if (live) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int i = 16 * kg + 4 * r + e;
                    const f32x4 v = f32x4{acc[e][0][r], acc[e][1][r], acc[e][2][r], acc[e][3][r]};
                    const uint32_t off = vu + ((I + 4 * r + e) * static_cast<uint32_t>(D) + J) * 4u;
                    if (!kDiag || 4 * row + 3 <= i) {
                        st_f32x4(Sb, off, v);
                    } else if (4 * row <= i) {
#pragma unroll
                        for (int f = 0; f < 4; ++f)
                            if (4 * row + f <= i)
                                *reinterpret_cast<float *>(reinterpret_cast<char *>(Sb) + off + 4 * f) = v[f];
                    }
                }
        }
    } else if constexpr (!kDiag) {
        if (live) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    st_f32x4(Sb, vu + ((I + 4 * r + e) * static_cast<uint32_t>(D) + J) * 4u,
                             f32x4{acc[e][0][r], acc[e][1][r], acc[e][2][r], acc[e][3][r]});
            // mirror, in two halves (f = 2h, 2h + 1) through the wave's LDS: lane (row, kg)
            // puts its 16-byte pieces of mirrored rows 4 row + f in place, then each store
            // writes four whole 256-byte rows (lane L: row 4 (L / 16) of the half, piece L % 16)
            float *w = tl + wave * kHalf;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
#pragma unroll
                for (int fo = 0; fo < 2; ++fo)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int f = 2 * h + fo;
                        *reinterpret_cast<f32x4 *>(w + (2 * row + fo) * (CT + 4) + 16 * kg + 4 * r) =
                            f32x4{acc[0][f][r], acc[1][f][r], acc[2][f][r], acc[3][f][r]};
                    }
                wave_lds_sync();
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    st_f32x4(Sb, vm + ((J + 8 * q + 2 * h) * static_cast<uint32_t>(D) + I) * 4u,
                             *reinterpret_cast<const f32x4 *>(w + (4 * q + (lane >> 4)) * (CT + 4) + 4 * (lane & 15)));
                wave_lds_sync();
            }
        }
    } else {
        float *w = tl + wave * CT * (CT + 1);
        if (live) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int f = 0; f < 4; ++f) w[(16 * kg + 4 * r + e) * (CT + 1) + 4 * row + f] = acc[e][f][r];
        }
        __syncthreads();
        if (live) {
            // entry (i, c) below the diagonal takes the value computed for (c, i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int i = 16 * kg + 4 * r + e;
                    f32x4 v;
#pragma unroll
                    for (int f = 0; f < 4; ++f)
                        v[f] = i > 4 * row + f ? w[(4 * row + f) * (CT + 1) + i] : acc[e][f][r];
                    st_f32x4(Sb, vu + ((I + 4 * r + e) * static_cast<uint32_t>(D) + I) * 4u, v);
                }
        }
    }
}

__global__ __launch_bounds__(256) void k_cov_f32(const float *g, int64_t ld, int B, int D, int nt,
                                                 float *S_all, bool lower) {
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
    add_and_mirror(S, D, I, J, ct, diag, lower);
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
    add_and_mirror(S, D, I, J, ct, diag, false);
}

}  // namespace

hipError_t launch_cov(const void *g, bool bf16, int64_t ld, int B, int D, int n_blocks, float *S, bool lower,
                      hipStream_t s) {
    if (B == 0 || n_blocks == 0) return hipSuccess;
    const int nt = (D + CT - 1) / CT;
    const dim3 grid(static_cast<unsigned>(nt * (nt + 1) / 2), static_cast<unsigned>(n_blocks));
    // register tiles: whole tiles, 8-byte row pieces, 128-bit S accesses, and
    // byte offsets of a block's S and of the rows within 32 bits
    const bool reg = D % CT == 0 && ld % 4 == 0 && (reinterpret_cast<uintptr_t>(g) & 7) == 0 &&
                     (reinterpret_cast<uintptr_t>(S) & 15) == 0 && D <= 16384 &&
                     (static_cast<int64_t>(B) + 32) * ld * 2 < (int64_t{1} << 31);
    const bf16_bits *gb = static_cast<const bf16_bits *>(g);
    if (bf16 && reg) {
        const int n_off = nt * (nt - 1) / 2;
        const dim3 off_grid(static_cast<unsigned>((n_off + 3) / 4), static_cast<unsigned>(n_blocks));
        if (n_off > 0) {
            if (lower)
                hipLaunchKernelGGL((k_cov_bf16_reg<false, true>), off_grid, dim3(256), 0, s, gb, ld, B, D, nt, n_off, S);
            else
                hipLaunchKernelGGL((k_cov_bf16_reg<false, false>), off_grid, dim3(256), 0, s, gb, ld, B, D, nt, n_off,
                                   S);
        }
        if (lower)
            hipLaunchKernelGGL((k_cov_bf16_reg<true, true>),
                               dim3(static_cast<unsigned>((nt + 3) / 4), static_cast<unsigned>(n_blocks)), dim3(256), 0,
                               s, gb, ld, B, D, nt, nt, S);
        else
            hipLaunchKernelGGL((k_cov_bf16_reg<true, false>),
                               dim3(static_cast<unsigned>((nt + 1) / 2), static_cast<unsigned>(n_blocks)), dim3(128), 0,
                               s, gb, ld, B, D, nt, nt, S);
    } else if (bf16) {
        hipLaunchKernelGGL(k_cov_bf16, grid, dim3(256), 0, s, gb, ld, B, D, nt, S, lower);
    } else {
        hipLaunchKernelGGL(k_cov_f32, grid, dim3(256), 0, s, static_cast<const float *>(g), ld, B, D, nt, S,
                           lower);
    }
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
