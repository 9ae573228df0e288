// PCA initialisation of the projections (Sec. 3.2): KFAC approximates a
// layer's Hessian block by C_F (x) C_B, the Kronecker product of the
// uncentered covariances of its forward activations and of its backward
// output gradients; P_i and P_o are initialised with the top-k_i and top-k_o
// eigenvectors of C_F and C_B.
//
// Activation covariance (SYRK):  C[i][j] += sum over unmasked tokens a_t[i] a_t[j]
//
//  0. k_slab_prep: lists the 32-token slabs (32 consecutive tokens of one
//     example) that hold at least one unmasked token, each with the 32-bit
//     map of its unmasked tokens.
//  1. k_act_cov_dma (bf16): one workgroup per upper-triangle 256 x 256 tile
//     (I <= J) of C; 4 waves, each owning a 128 x 128 quadrant as 4 x 4
//     blocks of 32x32x16 bf16 MFMAs (fp32 accumulation).  The contraction
//     runs over the listed slabs.  A slab of the two operands (the tile's
//     256 features I.. and J.. of 32 tokens, 16 KB each in token-major
//     order) is copied straight from memory into an LDS ring (gfx950
//     buffer_load ... lds), three slabs ahead; a masked token's row is read
//     as zeros without a memory access.  The MFMA operands need 8
//     consecutive tokens of one feature, so each fragment is gathered from
//     the token-major slab with 16-bit LDS reads.  A diagonal tile has one
//     operand.  The tile is added to C (upper part) and written mirrored to
//     the lower part, so C stays exactly symmetric.
//  1'. k_act_cov_f32: fp32 activations (small problems), one thread per entry.
//
// Every sum has a fixed order, so results are bitwise reproducible.
#include "common.h"
#include "internal.h"

namespace logra {
namespace {

constexpr int ST = 32;                          // tokens per slab
constexpr int CT = 256;                         // tile edge (features)
constexpr int kCSlab = ST * CT * 2;             // bytes of one operand slab (16 KB)
constexpr int kCStages = 4;                     // ring stages (slabs); each holds both operands
constexpr int kCStage = 2 * kCSlab;
constexpr int kCRow = CT + 1;                   // padded row of the epilogue's staging (floats)
constexpr int kCLds = 128 * kCRow * 4;          // >= ring (128 KB): the epilogue stages 128 rows
static_assert(kCStages * kCStage <= kCLds, "ring must fit the LDS allocation");
constexpr int kCCopies = kCSlab / 1024 / 4;     // 1 KB copies per wave and operand slab (4)

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

// Slabs of B examples of T tokens (spe = ceil(T / 32) per example): the
// non-empty ones in order, with bit r of bits[] set iff token 32 s + r of the
// example exists and is unmasked.  One workgroup, block-wide prefix counts.
__global__ __launch_bounds__(1024) void k_slab_prep(const uint8_t *mask, int B, int T, int spe, int *slabs,
                                                     uint32_t *bits, int *n_slabs) {
    __shared__ int wsum[16];
    __shared__ int base;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) base = 0;
    __syncthreads();
    const int total = B * spe;
    for (int s0 = 0; s0 < total; s0 += 1024) {
        const int sid = s0 + tid;
        uint32_t m = 0;
        if (sid < total) {
            const int b = sid / spe, t0 = (sid - b * spe) * ST;
            const int nv = min(ST, T - t0);
            for (int r = 0; r < nv; ++r)
                if (mask == nullptr || mask[static_cast<size_t>(b) * T + t0 + r] != 0) m |= 1u << r;
        }
        const int any = m != 0;
        int x = any;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(x, o, 64);
            if (lane >= o) x += y;
        }
        if (lane == 63) wsum[wave] = x;
        __syncthreads();
        int before = 0, all = 0;
        for (int w = 0; w < 16; ++w) {
            before += w < wave ? wsum[w] : 0;
            all += wsum[w];
        }
        if (any) {
            slabs[base + before + x - 1] = sid;
            bits[base + before + x - 1] = m;
        }
        __syncthreads();
        if (tid == 0) base += all;
        __syncthreads();
    }
    if (tid == 0) *n_slabs = base;
}

template <bool DIAG>
__device__ __forceinline__ void act_cov_tile(const bf16_bits *__restrict__ a, int T, int n, int spe,
                                             const int *__restrict__ slabs, const uint32_t *__restrict__ bits,
                                             int ns, int I, int J, float *__restrict__ C, uint8_t *smem) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const uint32_t lds0 = lds_addr(smem);
    constexpr int NOP = DIAG ? 1 : 2;               // operand slabs copied per slab
    constexpr int NCP = NOP * kCCopies;             // copies per wave per slab

    // copy q of this wave: token rows 2 (4 wave + q) + (lane >> 5) of the slab,
    // LDS chunk position lane & 31 of the row, holding feature chunk
    // (lane & 31) ^ (4 ((row >> 3) & 1)) (tokens r and r + 8 land 64 bytes
    // apart in the banks, so the fragment reads of the two half-waves do not
    // collide)
    int crow[kCCopies];
    uint32_t cofs[kCCopies];   // byte offset of the lane's 16 bytes within a token row, from feature 0
#pragma unroll
    for (int q = 0; q < kCCopies; ++q) {
        crow[q] = 2 * (4 * wave + q) + (lane >> 5);
        cofs[q] = static_cast<uint32_t>(((lane & 31) ^ (4 * ((crow[q] >> 3) & 1))) * 16);
    }
    auto issue = [&](int s, int stage) {
        const bool live = s < ns;
        const int sid = live ? slabs[s] : 0;
        const uint32_t m = live ? bits[s] : 0u;
        const int b = sid / spe, t0 = (sid - b * spe) * ST;
        const int rows = min(ST, T - t0);
        const bf16_bits *base = a + (static_cast<size_t>(b) * T + t0) * n;
        const auto rs = buf_rsrc_uniform(base, live ? static_cast<uint32_t>(rows * n * 2) : 0u);
        const uint32_t st = lds0 + stage * kCStage + wave * kCCopies * 1024;
#pragma unroll
        for (int o = 0; o < NOP; ++o) {
            const uint32_t f0 = static_cast<uint32_t>((o == 0 ? I : J) * 2);
#pragma unroll
            for (int q = 0; q < kCCopies; ++q) {
                const bool ok = (m >> crow[q]) & 1u;
                const uint32_t off = static_cast<uint32_t>(crow[q]) * static_cast<uint32_t>(n * 2) + f0 + cofs[q];
                copy_to_lds(rs, ok ? off : kBufOOB, st + o * kCSlab + q * 1024);
            }
        }
    };

    // fragment of block i (32 features) for the 16-token step ks: lane l holds
    // feature (l % 32) of the block, tokens 16 ks + 8 (l / 32) + e, e < 8
    const int sx = lane >> 5;   // (token >> 3) & 1 of every token the lane reads
    uint32_t fa[4], fb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int fA = wm * 128 + i * 32 + (lane & 31), fB = wn * 128 + i * 32 + (lane & 31);
        fa[i] = static_cast<uint32_t>(8 * sx * 512 + (((fA >> 3) ^ (4 * sx)) * 16) + (fA & 7) * 2);
        fb[i] = static_cast<uint32_t>(8 * sx * 512 + (((fB >> 3) ^ (4 * sx)) * 16) + (fB & 7) * 2) +
                (DIAG ? 0u : static_cast<uint32_t>(kCSlab));
    }
    typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
    auto frag = [&](const uint8_t *stage, uint32_t off, int ks) {
        u16x8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = *reinterpret_cast<const uint16_t *>(stage + off + (16 * ks + e) * 512);
        return __builtin_bit_cast(bf16x8, v);
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // Slab s lives in stage s % 4.  Before slab s is read, the copies in
    // flight are those of slabs s + 1 and s + 2 (issued in the two previous
    // steps): waiting until at most 2 NCP remain completes slab s.  The
    // barrier also ends every wave's reads of stage (s - 1) % 4, which the
    // copies of slab s + 3, issued next, overwrite.
    issue(0, 0);
    issue(1, 1);
    issue(2, 2);
    for (int s = 0; s < ns; ++s) {
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(2 * NCP) : "memory");
        issue(s + 3, (s + 3) & 3);
        const uint8_t *stage = smem + (s & 3) * kCStage;
        // (the below-diagonal quadrant of a diagonal tile is computed too and
        // discarded: a branch around the products would copy the accumulators)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            bf16x8 xa[4], xb[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                xa[i] = frag(stage, fa[i], ks);
                xb[i] = frag(stage, fb[i], ks);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma32_bf16(xa[i], xb[j], acc[i][j]);
        }
    }
    // the copies past the last slab are still in flight
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");

    // Epilogue, one half of the tile's rows (wm = h) at a time: the owning
    // waves add their quadrants to C's upper part and stage the new values in
    // LDS; then all threads write them mirrored (rows of the mirror are
    // contiguous along the tile's rows).
    float *ct = reinterpret_cast<float *>(smem);
#pragma unroll 1
    for (int h = 0; h < 2; ++h) {
        if (wm == h) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                        const int col = wn * 128 + j * 32 + (lane & 31);
                        const int gi = I + h * 128 + row, gj = J + col;
                        if (gi < n && gj < n && (!DIAG || gi <= gj)) {
                            float *p = C + static_cast<size_t>(gi) * n + gj;
                            const float v = *p + acc[i][j][r];
                            *p = v;
                            ct[row * kCRow + col] = v;
                        }
                    }
        }
        __syncthreads();
        for (int e = tid; e < 128 * CT; e += 256) {
            const int col = e >> 7, row = e & 127;   // consecutive threads: consecutive rows
            const int gi = I + h * 128 + row, gj = J + col;
            if (gi < n && gj < n && (DIAG ? gi < gj : true))
                C[static_cast<size_t>(gj) * n + gi] = ct[row * kCRow + col];
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(256, 1) void k_act_cov_dma(const bf16_bits *__restrict__ a, int T, int n, int spe,
                                                        const int *__restrict__ slabs,
                                                        const uint32_t *__restrict__ bits,
                                                        const int *__restrict__ n_slabs, int nt,
                                                        float *__restrict__ C) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[kCLds];
    int ti, tj;
    tile_coords(blockIdx.x, nt, ti, tj);
    const int ns = __builtin_amdgcn_readfirstlane(*n_slabs);
    if (ti == tj)
        act_cov_tile<true>(a, T, n, spe, slabs, bits, ns, ti * CT, tj * CT, C, smem);
    else
        act_cov_tile<false>(a, T, n, spe, slabs, bits, ns, ti * CT, tj * CT, C, smem);
}

// fp32 activations: one thread per upper entry (i <= j) of a 16 x 16 block,
// summing over the listed slabs' unmasked tokens in order; both entries written.
__global__ __launch_bounds__(256) void k_act_cov_f32(const float *__restrict__ a, int T, int n, int spe,
                                                     const int *__restrict__ slabs,
                                                     const uint32_t *__restrict__ bits,
                                                     const int *__restrict__ n_slabs, float *__restrict__ C) {
    const int i = blockIdx.y * 16 + (threadIdx.x >> 4), j = blockIdx.x * 16 + (threadIdx.x & 15);
    if (i >= n || j >= n || i > j) return;
    const int ns = *n_slabs;
    float s = 0.f;
    for (int k = 0; k < ns; ++k) {
        const int sid = slabs[k];
        const uint32_t m = bits[k];
        const int b = sid / spe, t0 = (sid - b * spe) * ST;
        const float *row = a + (static_cast<size_t>(b) * T + t0) * n;
        for (int r = 0; r < ST; ++r)
            if ((m >> r) & 1u) s = __builtin_fmaf(row[static_cast<size_t>(r) * n + i], row[static_cast<size_t>(r) * n + j], s);
    }
    const float v = C[static_cast<size_t>(i) * n + j] + s;
    C[static_cast<size_t>(i) * n + j] = v;
    if (i != j) C[static_cast<size_t>(j) * n + i] = v;
}

}  // namespace

size_t act_cov_ws_bytes(int B, int T) {
    const size_t slabs = static_cast<size_t>(B) * ((T + ST - 1) / ST);
    return align256(sizeof(int) * slabs) + align256(sizeof(uint32_t) * slabs) + 256;
}

hipError_t launch_act_cov(const void *a, bool bf16, int B, int T, int n, const uint8_t *mask, float *C, void *ws,
                          hipStream_t s) {
    if (B == 0 || T == 0) return hipSuccess;
    const int spe = (T + ST - 1) / ST;
    const size_t slabs = static_cast<size_t>(B) * spe;
    char *w = static_cast<char *>(ws);
    int *list = reinterpret_cast<int *>(w);
    uint32_t *bits = reinterpret_cast<uint32_t *>(w + align256(sizeof(int) * slabs));
    int *count = reinterpret_cast<int *>(w + align256(sizeof(int) * slabs) + align256(sizeof(uint32_t) * slabs));
    hipLaunchKernelGGL(k_slab_prep, dim3(1), dim3(1024), 0, s, mask, B, T, spe, list, bits, count);
    if (bf16) {
        const int nt = (n + CT - 1) / CT;
        hipLaunchKernelGGL(k_act_cov_dma, dim3(static_cast<unsigned>(nt * (nt + 1) / 2)), dim3(256), 0, s,
                           static_cast<const bf16_bits *>(a), T, n, spe, list, bits, count, nt, C);
    } else {
        const unsigned nb = static_cast<unsigned>((n + 15) / 16);
        hipLaunchKernelGGL(k_act_cov_f32, dim3(nb, nb), dim3(256), 0, s, static_cast<const float *>(a), T, n, spe,
                           list, bits, count, C);
    }
    return hipGetLastError();
}

}  // namespace logra
