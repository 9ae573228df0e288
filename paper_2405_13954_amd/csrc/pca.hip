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
//     (I <= J) of C, tiles grouped per XCD for L2 reuse (one launch may hold
//     several factors of the same batch, each with a range of workgroup
//     slots); 4 waves, each owning a 128 x 128 quadrant as 4 x 4
//     blocks of 32x32x16 bf16 MFMAs (fp32 accumulation).  The contraction
//     runs over the listed slabs.  A slab of the two operands (the tile's
//     256 features I.. and J.. of 32 tokens, 16 KB each in token-major
//     order) is copied straight from memory into an LDS ring (gfx950
//     buffer_load ... lds), four slabs ahead; a masked token's row is read
//     as zeros without a memory access.  The MFMA operands need 8
//     consecutive tokens of one feature: each fragment is two transposed
//     LDS reads (gfx950 ds_read_b64_tr_b16) of the token-major slab.  A
//     diagonal tile has one operand.  The tile is staged in LDS, added to
//     C's upper part with coalesced read-modify-writes and written mirrored
//     to the lower part, so C stays exactly symmetric.
//  1'. k_act_cov_f32: fp32 activations (small problems), one thread per entry.
//
// Top-k eigenvectors of C (n x n, symmetric PSD, fp32), by subspace
// iteration on p = min(n, max(2k, 16)) vectors with Rayleigh-Ritz extraction:
//
//   Q_0 = a fixed pseudo-random n x p block;  repeat `iters` times:
//       Z = C Q  (fp32 MFMA, one pass over C);  Q = Z R^{-1}, R^T R = Z^T Z + eps
//   then once more with a second orthonormalisation (CholQR2), T = Q^T C Q,
//   T = W diag(theta) W^T (cyclic Jacobi, fp64), and the Ritz vectors
//   v_e = Q w_e of the k largest theta, each signed so that its entry of
//   largest magnitude (lowest index among equal magnitudes) is positive.
//
//  Q and Z are kept in row quads (four rows of a column adjacent).
//  2. k_cq_dma / k_cq_regs (+ k_cq_sum): Z = C Q; a workgroup owns 64 rows
//     of C (32 for p > 64) and a range of its columns, its waves splitting
//     the range; 16x16x4 fp32 MFMAs.  p <= 64 (bound by the reads of C):
//     64-column slabs of C and Q copied into an LDS ring; wider: 128-bit
//     loads into a register pipeline.  Column ranges (splits) give about
//     2048 workgroups; their partials are summed in split order.
//  3. k_gram_part: fp64 partial sums of X^T Y over 64-row chunks (X^T X for
//     the orthonormalisation, Z^T Q for Rayleigh-Ritz), fixed order.
//  4. k_chol_inv_cols (one workgroup): the chunk sums (summed on the chip
//     first by k_sum_parts), a shifted Cholesky Z^T Z + eps tr/p I =
//     R^T R and R^{-1} in fp64, columns in registers and each step's row
//     broadcast through LDS (p <= 64: one wave; wider: four waves, one
//     barrier per step).
//  5. k_apply_rinv: Q = Z R^{-1} (fp64 arithmetic, fp32 result).
//  6. k_jacobi_rot (one workgroup): T in LDS, round-robin parallel cyclic
//     Jacobi (m/2 disjoint rotations per round, each round one pass of 2 x 2
//     blocks), the rotations logged; k_jacobi_replay: W^T = the logged
//     rotations applied to the identity, one wave per column.
//  7. k_ritz, k_pca_out: Ritz vectors in the order of decreasing theta, the
//     sign rule, and the rows of P in the output dtype.
//
// Every sum has a fixed order, so results are bitwise reproducible.
#include <algorithm>
#include <cstdint>
#include <utility>

#include "common.h"
#include "internal.h"

namespace logra {
namespace {

constexpr int ST = 32;                          // tokens per slab
constexpr int CT = 256;                         // tile edge (features)
constexpr int kCSlab = ST * CT * 2;             // bytes of one operand slab (16 KB)
constexpr int kCStages = 5;                     // ring stages (slabs); each holds both operands
constexpr int kCStage = 2 * kCSlab;
constexpr int kCRow = CT + 1;                   // padded row of the epilogue's staging (floats)
constexpr int kCLds = kCStages * kCStage;       // 160 KB
static_assert(128 * kCRow * 4 <= kCLds, "the epilogue stages 128 rows of a tile in the ring");
constexpr int kGR = 4, kGC = 8;                 // tiles per XCD group: 4 tile rows x 8 tile columns
constexpr int kCCopies = kCSlab / 1024 / 4;     // 1 KB copies per wave and operand slab (4)

// Tile of workgroup `bid`, grouped for the L2 caches.  Dispatch deals
// workgroups round-robin over the 8 XCDs (bid % 8) and one workgroup fills a
// CU, so each XCD runs 32 at a time.  They get a group of 4 tile rows x 8 tile
// columns, which reads 12 distinct 256-feature blocks of the activations
// instead of 64, in step (same slabs at about the same time).  Groups holding
// an upper-triangle tile are numbered row by row (group row gr starts at
// group column gr / 2) and dealt to XCDs in turn.  Returns false for a slot
// with no upper tile.
__device__ __forceinline__ bool tile_of(int bid, int nt, int &ti, int &tj) {
    const int x = bid & 7, u = bid >> 3;
    int g = (u / (kGR * kGC)) * 8 + x;
    const int slot = u % (kGR * kGC);
    const int ngr = (nt + kGR - 1) / kGR, ngc = (nt + kGC - 1) / kGC;
    int gr = 0;
    while (gr < ngr && g >= ngc - gr / 2) {
        g -= ngc - gr / 2;
        ++gr;
    }
    if (gr >= ngr) return false;
    ti = gr * kGR + slot / kGC;
    tj = (gr / 2 + g) * kGC + slot % kGC;
    return ti < nt && tj < nt && ti <= tj;
}

inline int tile_slots(int nt) {
    const int ngr = (nt + kGR - 1) / kGR, ngc = (nt + kGC - 1) / kGC;
    int groups = 0;
    for (int gr = 0; gr < ngr; ++gr) groups += ngc - gr / 2;
    return (groups + 7) / 8 * 8 * kGR * kGC;
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

    // LDS slab layout: 32 token rows of 512 bytes (the tile's 256 features);
    // the 16-byte chunk c of token row t sits at position c ^ (4 (t & 3)), so
    // that the four token rows read together by a transposed read (below)
    // fall in different banks.  Copy q of this wave fills token rows
    // 2 (4 wave + q) + (lane >> 5): lane l stores position l & 31 of its row.
    int crow[kCCopies];
    uint32_t cofs[kCCopies];   // byte offset of the lane's 16 bytes within a token row, from feature 0
#pragma unroll
    for (int q = 0; q < kCCopies; ++q) {
        crow[q] = 2 * (4 * wave + q) + (lane >> 5);
        cofs[q] = static_cast<uint32_t>(((lane & 31) ^ (4 * (crow[q] & 3))) * 16);
    }
    // copy c (< NCP) of a slab: operand c / 4 (I, then J), copy c % 4 of the wave
    struct Slab {
        __amdgpu_buffer_rsrc_t rs;
        uint32_t m;
    };
    auto slab_of = [&](int sid, uint32_t m) {
        const int b = sid / spe, t0 = (sid - b * spe) * ST;
        const int rows = min(ST, T - t0);
        const bf16_bits *base = a + (static_cast<size_t>(b) * T + t0) * n;
        return Slab{buf_rsrc_uniform(base, m ? static_cast<uint32_t>(rows * n * 2) : 0u), m};
    };
    auto copy1 = [&](const Slab &sl, int stage, int c) {
        const int o = c / kCCopies, q = c % kCCopies;
        const uint32_t f0 = static_cast<uint32_t>((o == 0 ? I : J) * 2);
        const bool ok = (sl.m >> crow[q]) & 1u;
        const uint32_t off = static_cast<uint32_t>(crow[q]) * static_cast<uint32_t>(n * 2) + f0 + cofs[q];
        copy_to_lds(sl.rs, ok ? off : kBufOOB,
                    lds0 + stage * kCStage + o * kCSlab + wave * kCCopies * 1024 + q * 1024);
    };

    // MFMA fragment of block i (32 features) for the 16-token step ks: lane l
    // must hold feature l % 32 of the block and tokens 16 ks + 8 (l / 32) + 0..7.
    // A transposed LDS read (ds_read_b64_tr_b16) works on groups of 16 lanes:
    // slot e of lane i receives element i % 4 of the 8 bytes addressed by lane
    // 4 e + i / 4.  So lane j of group g (= l / 16) addresses token
    // 16 ks + 8 (g / 2) + 4 r + j / 4, features (g % 2) 16 + 4 (j % 4) .. + 3 of
    // the block, and read r (0, 1) hands every lane tokens 4 r .. 4 r + 3 of
    // its feature.
    const int gq = lane >> 4, jq = lane & 15;
    uint32_t fa[4], fb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int t = 8 * (gq >> 1) + (jq >> 2);                    // token within the step, r = 0
        const int fA = wm * 128 + i * 32 + (gq & 1) * 16 + 4 * (jq & 3);
        const int fB = wn * 128 + i * 32 + (gq & 1) * 16 + 4 * (jq & 3);
        fa[i] = static_cast<uint32_t>(t * 512 + (((fA >> 3) ^ (4 * (t & 3))) * 16) + (fA & 7) * 2);
        fb[i] = static_cast<uint32_t>(t * 512 + (((fB >> 3) ^ (4 * (t & 3))) * 16) + (fB & 7) * 2) +
                (DIAG ? 0u : static_cast<uint32_t>(kCSlab));
    }
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    bf16x8 xa[2][4], xb[2][4];   // fragments: buffer 0 for the step ks = 0, buffer 1 for ks = 1
    // fragment q of a step: A block q for q < 4, B block q - 4 otherwise
    auto ldfrag = [&](int buf, uint32_t stage_off, int ks, int q) {
        const uint32_t p0 = lds0 + stage_off + (q < 4 ? fa[q] : fb[q - 4]) + static_cast<uint32_t>(16 * ks * 512);
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(uintptr_t)p0);
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(uintptr_t)(p0 + 4 * 512));
        const s16x4 v8[2] = {lo, hi};
        const bf16x8 v = __builtin_bit_cast(bf16x8, v8);
        if (q < 4)
            xa[buf][q] = v;
        else
            xb[buf][q - 4] = v;
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    auto mfma1 = [&](int buf, int idx) {
        const int i = idx >> 2, j = idx & 3;
        acc[i][j] = mfma32_bf16(xa[buf][i], xb[buf][j], acc[i][j]);
    };

    // Slab s lives in stage s % 5; the copies of slab s + 4 go to stage
    // (s - 1) % 5 while slab s is multiplied (that stage's last reads, the
    // fragments of slab s - 1, completed before the previous barrier).  The
    // step ks = 0 of a slab reads the fragments of its step ks = 1 and
    // issues the copies; the barrier sits in the middle of step ks = 1, after
    // each wave has waited for its copies of slab s + 1 (at most the three
    // later slabs' copies in flight) and its fragment reads; the second half
    // of step ks = 1 reads the fragments of slab s + 1's step ks = 0.  The
    // order is fixed (scheduling barriers): groups of MFMAs with one
    // fragment and one copy.  The list entry of a slab is loaded one step
    // before its copies are issued.  (The below-diagonal quadrant of a
    // diagonal tile is computed and discarded: a branch around the products
    // would copy the accumulators.)
    auto entry = [&](int s, int &sid, uint32_t &m) {
        sid = s < ns ? slabs[s] : 0;
        m = s < ns ? bits[s] : 0u;
    };
    {
        int sid;
        uint32_t m;
#pragma unroll
        for (int s = 0; s < kCStages - 1; ++s) {
            entry(s, sid, m);
            const Slab sl = slab_of(sid, m);
#pragma unroll
            for (int c = 0; c < NCP; ++c) copy1(sl, s, c);
        }
    }
    int nsid;
    uint32_t nm;
    entry(kCStages - 1, nsid, nm);
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" :: "n"((kCStages - 2) * NCP) : "memory");
#pragma unroll
    for (int q = 0; q < 8; ++q) ldfrag(0, 0u, 0, q);
    int cur = 0, nxt = kCStages - 1;   // stages of slab s and of slab s + 4
    for (int s = 0; s < ns; ++s) {
        const Slab sl = slab_of(nsid, nm);
        entry(s + kCStages, nsid, nm);
        const uint32_t cur_off = static_cast<uint32_t>(cur * kCStage);
        const int nc = cur == kCStages - 1 ? 0 : cur + 1;   // stage of slab s + 1
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            mfma1(0, 2 * q);
            mfma1(0, 2 * q + 1);
            ldfrag(1, cur_off, 1, q);
            if (q < NCP) copy1(sl, nxt, q);
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) mfma1(1, q);
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"((kCStages - 2) * NCP) : "memory");
        const uint32_t next_off = static_cast<uint32_t>(nc * kCStage);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            ldfrag(0, next_off, 0, q);
            mfma1(1, 8 + q);
            __builtin_amdgcn_sched_barrier(0);
        }
        cur = nc;
        nxt = nxt == kCStages - 1 ? 0 : nxt + 1;
    }
    // the copies past the last slab are still in flight
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");

    // Epilogue, one half of the tile's rows (wm = h) at a time: the owning
    // waves stage their quadrants in LDS; all threads then add the staged
    // rows to C's upper part (coalesced 16-byte read-modify-writes, the new
    // values written back to the staging) and write them mirrored (rows of
    // the mirror run along the tile's rows).
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
                        ct[row * kCRow + col] = acc[i][j][r];
                    }
        }
        __syncthreads();
        // Read-modify-write in batches of kBatch quads per thread, every load
        // of a batch issued before its first store: a store to C might alias
        // a later load, so the compiler would otherwise keep each load behind
        // the previous store, one memory round trip per quad.
        constexpr int kQuads = 128 * (CT / 4) / 256, kBatch = 16;
#pragma unroll
        for (int b0 = 0; b0 < kQuads; b0 += kBatch) {
            f32x4 old[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int e = tid + 256 * (b0 + u);
                const int row = e / (CT / 4), c4 = 4 * (e % (CT / 4));
                const int gi = I + h * 128 + row, gj = J + c4;
                const float *p = C + static_cast<size_t>(gi) * n + gj;
                old[u] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (gi >= n) continue;
                if (gj + 3 < n && (!DIAG || gi <= gj)) {
                    old[u] = *reinterpret_cast<const f32x4 *>(p);
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        if (gj + k < n && (!DIAG || gi <= gj + k)) old[u][k] = p[k];
                }
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int e = tid + 256 * (b0 + u);
                const int row = e / (CT / 4), c4 = 4 * (e % (CT / 4));
                const int gi = I + h * 128 + row, gj = J + c4;
                if (gi >= n) continue;
                float *p = C + static_cast<size_t>(gi) * n + gj;
                float *st = ct + row * kCRow + c4;
                if (gj + 3 < n && (!DIAG || gi <= gj)) {
                    const f32x4 v = old[u] + f32x4{st[0], st[1], st[2], st[3]};
                    *reinterpret_cast<f32x4 *>(p) = v;
#pragma unroll
                    for (int k = 0; k < 4; ++k) st[k] = v[k];
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        if (gj + k < n && (!DIAG || gi <= gj + k)) {
                            const float v = old[u][k] + st[k];
                            p[k] = v;
                            st[k] = v;
                        }
                }
            }
        }
        __syncthreads();
        // The mirror: four consecutive rows of one column per thread, one
        // 16-byte store where all four belong below the diagonal and in range.
        for (int e = tid; e < 32 * CT; e += 256) {
            const int col = e >> 5, q = e & 31;   // consecutive threads: consecutive row quads
            const int gi = I + h * 128 + 4 * q, gj = J + col;
            if (gj >= n) continue;
            const float *sv = ct + 4 * q * kCRow + col;
            float *dst = C + static_cast<size_t>(gj) * n + gi;
            if (gi + 3 < n && (!DIAG || gi + 3 < gj)) {
                *reinterpret_cast<f32x4 *>(dst) = f32x4{sv[0], sv[kCRow], sv[2 * kCRow], sv[3 * kCRow]};
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (gi + k < n && (!DIAG || gi + k < gj)) dst[k] = sv[k * kCRow];
            }
        }
        __syncthreads();
    }
}

// The factors of one launch: factor f owns the workgroup slots
// [slot_end[f - 1], slot_end[f]) (tile_slots of its tile count, a multiple of
// 256, so a slot's XCD is the same as in a launch of its own).
struct ActCovFactor {
    const bf16_bits *a;
    float *C;
    int n, nt, slot_end;
};
struct ActCovArgs {
    ActCovFactor f[kMaxActCovGroup];
    int count;
};

__global__ __launch_bounds__(256, 1) void k_act_cov_dma(ActCovArgs g, int T, int spe,
                                                        const int *__restrict__ slabs,
                                                        const uint32_t *__restrict__ bits,
                                                        const int *__restrict__ n_slabs) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[kCLds];
    const int bid = blockIdx.x;
    int f = 0;
    while (f + 1 < g.count && bid >= g.f[f].slot_end) ++f;
    const ActCovFactor &F = g.f[f];
    int ti, tj;
    if (!tile_of(bid - (f > 0 ? g.f[f - 1].slot_end : 0), F.nt, ti, tj)) return;
    const int ns = __builtin_amdgcn_readfirstlane(*n_slabs);
    if (ti == tj)
        act_cov_tile<true>(F.a, T, F.n, spe, slabs, bits, ns, ti * CT, tj * CT, F.C, smem);
    else
        act_cov_tile<false>(F.a, T, F.n, spe, slabs, bits, ns, ti * CT, tj * CT, F.C, smem);
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

// ------------------------------------------------------------------------
// Subspace iteration for the top-k eigenvectors.
//
// Q and Z (n x pp fp32; pp = p rounded up to 16) are stored in row quads:
// element (i, j) at ((i / 4) pp + j) 4 + i % 4, with the rows padded to
// n4 = n rounded up to 4 and every element past n or p zero.  Four
// consecutive rows of one column (the B operand of a 16x16x4 MFMA) are then
// one 128-bit load, and a run of rows is one contiguous range.
constexpr int kGramRows = 64;    // rows per partial sum of a Gram matrix
constexpr int kGramChunk = 64;   // rows staged in LDS at a time
constexpr int kMaxP = 128;       // subspace width (at most 2 k for k <= 64)
constexpr int kCqStages = 3;     // register pipeline depth of k_cq_regs
constexpr int kJacobiSweeps = 40;   // at most this many Jacobi sweeps

__host__ __device__ constexpr int round4(int n) { return (n + 3) & ~3; }
__device__ __forceinline__ size_t qidx(int i, int j, int pp) {
    return ((static_cast<size_t>(i >> 2) * pp + j) << 2) + (i & 3);
}

__device__ __forceinline__ float hash_uniform(uint32_t i, uint32_t j) {
    // integer hash of (i, j) (a multiply-xorshift mixer) -> uniform in [-1, 1)
    uint32_t h = i * 0x9E3779B1u ^ (j + 0x7F4A7C15u) * 0x85EBCA77u;
    h ^= h >> 16;
    h *= 0x7FEB352Du;
    h ^= h >> 15;
    h *= 0x846CA68Bu;
    h ^= h >> 16;
    return static_cast<float>(h >> 8) * (2.0f / 16777216.0f) - 1.0f;
}

// Q_0: pseudo-random columns j < p, zeros elsewhere (row quads, n4 rows).
__global__ __launch_bounds__(256) void k_pca_init(float *Q, int n, int p, int pp) {
    const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (e >= static_cast<int64_t>(round4(n)) * pp) return;
    const int64_t qj = e >> 2;
    const int i = static_cast<int>(qj / pp) * 4 + static_cast<int>(e & 3);
    const int j = static_cast<int>(qj % pp);
    Q[e] = i < n && j < p ? hash_uniform(static_cast<uint32_t>(i), static_cast<uint32_t>(j)) : 0.f;
}

// The end of both C Q kernels: fold the four waves' sums ((w3 + w2) + w1) +
// w0 through LDS (`fold`, MR NB 64 128-bit slots) and store the result in row
// quads to Z (one split) or the split's partial.  Result register r of lane
// (row, q) is row 4 q + r, column row of its 16 x 16 block: four consecutive
// rows of one column, one 128-bit store.
template <int NB, int MR>
__device__ __forceinline__ void cq_fold_store(const f32x4 (&acc)[MR][NB], f32x4 *fold, int lane, int wave, int m0,
                                              int n4, float *__restrict__ Zs) {
    constexpr int pp = 16 * NB;
    const int row = lane & 15, q = lane >> 4;
    f32x4 *my = fold + lane;
    if (wave == 3) {
#pragma unroll
        for (int m = 0; m < MR; ++m)
#pragma unroll
            for (int b = 0; b < NB; ++b) my[(m * NB + b) * kWave] = acc[m][b];
    }
    __syncthreads();
#pragma unroll
    for (int w = 2; w >= 1; --w) {
        if (wave == w) {
#pragma unroll
            for (int m = 0; m < MR; ++m)
#pragma unroll
                for (int b = 0; b < NB; ++b) my[(m * NB + b) * kWave] = my[(m * NB + b) * kWave] + acc[m][b];
        }
        __syncthreads();
    }
    if (wave == 0) {
        float *dst = Zs + static_cast<size_t>(blockIdx.y) * n4 * pp;
#pragma unroll
        for (int m = 0; m < MR; ++m) {
            const int i0 = m0 + 16 * m + 4 * q;
            if (i0 >= n4) continue;
#pragma unroll
            for (int b = 0; b < NB; ++b)
                *reinterpret_cast<f32x4 *>(dst + qidx(i0, 16 * b + row, pp)) =
                    my[(m * NB + b) * kWave] + acc[m][b];
        }
    }
}

// Z_s = C[:, K_s] Q[K_s, :] over the column range K_s = [s kr, (s + 1) kr) of
// split s = blockIdx.y (kr a multiple of 64).  A workgroup owns R = 16 MR
// rows of C and streams the range in 64-column slabs: each slab's R rows of
// C (256 bytes per row, whole cache lines) and the 16 row quads of Q it
// meets are copied straight into an LDS ring by asynchronous global-to-LDS
// copies, one slab ahead: two stages (48 KB at p = 32) let three workgroups
// share a CU, whose copies overlap one another's MFMAs (at n = 14336, p = 32:
// 154 us per pass; three stages and two workgroups 170 us; four stages and
// one workgroup slower still).  Wave w takes the slab's 16-column step w: lane
// (row, q) reads columns 4q .. 4q + 3 of that step in each row block and rows
// 4q .. 4q + 3 of one column of each 16-column block of Q (one 128-bit LDS
// read each; C's 16-byte chunks sit at chunk ^ (row & 15), so the reads of a
// row block hit 16 different bank groups), and feeds them to 16x16x4 fp32
// MFMAs, element e of both to MFMA e.  So wave w sums the range's steps w,
// w + 4, ... in order.  The waves' sums are folded in a fixed order through
// LDS and written, in row quads, to Z (one split) or to the split's partial.
// Rows past n read zeros; so do columns past the range's end; columns past n
// meet the zero rows of Q past n (a chunk straddling the end of a row reads
// the next row's first columns, or zeros past the end of C, against those
// zeros).  Every memory operation in the loop is a copy, so waiting until
// only the later slabs' copies are pending is exact.
template <int NB, int MR>
struct CqDma {
    static constexpr int R = 16 * MR, PP = 16 * NB;
    static constexpr int kC = R * 256;              // bytes of a slab's rows of C
    static constexpr int kQ = 16 * PP * 16;         // bytes of its 16 row quads of Q
    static constexpr int kStage = kC + kQ;
    static constexpr int kStages = 2;
    static constexpr int kCopies = (kC + kQ) / 1024 / 4;   // 1 KB copies per wave per slab (MR + NB)
    static_assert(kCopies == MR + NB, "each wave copies MR row groups of C and NB kilobytes of Q");
    static_assert(MR * NB * kWave * 16 <= kStage, "the fold fits in one stage");
};

template <int NB, int MR>
__global__ __launch_bounds__(256) void k_cq_dma(const float *__restrict__ C, int n, const float *__restrict__ Q,
                                                int kr, float *__restrict__ Zs) {
    using Sh = CqDma<NB, MR>;
    constexpr int NS = Sh::kStages, pp = Sh::PP;
    __shared__ __attribute__((aligned(1024))) uint8_t ring[NS * Sh::kStage];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int row = lane & 15, q = lane >> 4;
    const int m0 = blockIdx.x * Sh::R;
    const int k0 = blockIdx.y * kr;
    const int k1 = min(n, k0 + kr);
    const int n4 = round4(n);
    const int rows = min(Sh::R, n - m0);
    const auto rc = buf_rsrc_uniform(C + static_cast<size_t>(m0) * n, static_cast<uint32_t>(rows) * n * 4u);
    const auto rq = buf_rsrc_uniform(Q, static_cast<uint32_t>(n4) * pp * 4u);
    const uint32_t lds0 = lds_addr(ring);
    // copy i of this wave (i < MR) covers slab rows 4 (MR wave + i) .. + 3:
    // lane l writes position l & 15 of row 4 (MR wave + i) + (l >> 4), which
    // holds the row's chunk (l & 15) ^ (row & 15)
    uint32_t coff[MR];
    int ccol[MR];
#pragma unroll
    for (int i = 0; i < MR; ++i) {
        const int r = 4 * (MR * wave + i) + (lane >> 4);
        ccol[i] = 4 * ((lane & 15) ^ (r & 15));
        coff[i] = r < rows ? static_cast<uint32_t>(r * n + ccol[i]) * 4u : kBufOOB;
    }
    // copy i of this wave (i < NB) covers kilobyte NB wave + i of the slab's Q quads
    const uint32_t qoff = static_cast<uint32_t>(NB * wave) * 1024u + static_cast<uint32_t>(lane) * 16u;
    const int nslabs = (k1 - k0 + 63) / 64;
    auto issue = [&](int sl, int stage) {   // slabs past the range: all out of range
        const int k = k0 + 64 * sl;
        const uint32_t lds = lds0 + static_cast<uint32_t>(stage * Sh::kStage);
#pragma unroll
        for (int i = 0; i < MR; ++i) {
            const bool in = sl < nslabs && k + ccol[i] < k1;
            copy_to_lds(rc, in ? coff[i] + static_cast<uint32_t>(k) * 4u : kBufOOB,
                        lds + static_cast<uint32_t>(MR * wave + i) * 1024u);
        }
        const uint32_t kq = static_cast<uint32_t>(k) * pp * 4u;   // bytes of row quad k / 4
#pragma unroll
        for (int i = 0; i < NB; ++i)
            copy_to_lds(rq, sl < nslabs ? kq + qoff + static_cast<uint32_t>(i) * 1024u : kBufOOB,
                        lds + static_cast<uint32_t>(Sh::kC + (NB * wave + i) * 1024));
    };

    f32x4 acc[MR][NB];
#pragma unroll
    for (int m = 0; m < MR; ++m)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[m][b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < NS - 1; ++i) issue(i, i);
    const int cpos = ((4 * wave + q) ^ row) * 16;   // this lane's chunk within a row of its row blocks
    for (int sl = 0; sl < nslabs; ++sl) {
        // this wave's copies of slab sl are done when at most the NS - 2 later
        // slabs' copies are pending; after the barrier every wave's are, and
        // every wave has read slab sl - 1, whose stage the next copies refill
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"((NS - 2) * Sh::kCopies) : "memory");
        issue(sl + NS - 1, (sl + NS - 1) % NS);
        const uint8_t *cb = ring + (sl % NS) * Sh::kStage;
        const uint8_t *qb = cb + Sh::kC;
        u32x4 cv[MR], qv[NB];
#pragma unroll
        for (int m = 0; m < MR; ++m) cv[m] = *reinterpret_cast<const u32x4 *>(cb + (16 * m + row) * 256 + cpos);
#pragma unroll
        for (int b = 0; b < NB; ++b)
            qv[b] = *reinterpret_cast<const u32x4 *>(qb + ((4 * wave + q) * pp + 16 * b + row) * 16);
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int m = 0; m < MR; ++m)
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    acc[m][b] = mfma16_f32(__uint_as_float(cv[m][e]), __uint_as_float(qv[b][e]), acc[m][b]);
    }
    // the copies past the range (zeros) are still in flight; stage 0 then
    // holds the fold
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    cq_fold_store<NB, MR>(acc, reinterpret_cast<f32x4 *>(ring), lane, wave, m0, n4, Zs);
}

// Z_s = C[:, K_s] Q[K_s, :] as k_cq_dma computes it (the same steps, sums
// and fold), for wide subspaces (pp > 64).  There the 16x16x4 fp32 MFMAs,
// not the reads of C, bound the pass, and an LDS ring would leave room for
// one workgroup per CU; the waves of several workgroups hide the MFMA and
// load latencies better.  A workgroup owns 16 MR rows of C; its four waves
// take the range's 16-column steps round-robin.  Lane (row, q) of a wave
// streams columns k + 4q .. k + 4q + 3 of its row in each row block (one
// 128-bit load per block) and rows k + 4q .. k + 4q + 3 of one column of
// each 16-column block of Q (one 128-bit load), and feeds them to the
// MFMAs, element e of both to MFMA e.  A register pipeline keeps
// kCqStages - 1 steps in flight; every load is unconditional (out-of-range
// offsets read zeros).  Rows past n read zeros; columns past n meet the zero
// rows of Q past n (a load straddling the end of a row reads the next row's
// first columns, or zeros past the end of C, against those zeros).
template <int NB, int MR>
__global__ __launch_bounds__(256) void k_cq_regs(const float *__restrict__ C, int n, const float *__restrict__ Q,
                                                 int kr, float *__restrict__ Zs) {
    constexpr int pp = 16 * NB;
    constexpr int ST = kCqStages;
    __shared__ f32x4 fold[MR * NB * kWave];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int row = lane & 15, q = lane >> 4;
    const int m0 = blockIdx.x * 16 * MR;
    const int k0 = blockIdx.y * kr;
    const int k1 = min(n, k0 + kr);
    const int n4 = round4(n);
    const int rows = min(16 * MR, n - m0);
    const auto rc = buf_rsrc_uniform(C + static_cast<size_t>(m0) * n, static_cast<uint32_t>(rows) * n * 4u);
    const auto rq = buf_rsrc_uniform(Q, static_cast<uint32_t>(n4) * pp * 4u);
    uint32_t coff[MR];
#pragma unroll
    for (int m = 0; m < MR; ++m)
        coff[m] = 16 * m + row < rows ? (static_cast<uint32_t>(16 * m + row) * n + 4 * q) * 4u : kBufOOB;
    const uint32_t qoff = static_cast<uint32_t>(q * pp + row) * 16u;   // bytes of Q's element (4 q, row)

    f32x4 acc[MR][NB];
#pragma unroll
    for (int m = 0; m < MR; ++m)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[m][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int nsteps = (k1 - k0 + 15) / 16;
    if (wave < nsteps) {
        auto load = [&](int st, u32x4(&cv)[MR], u32x4(&qv)[NB]) {
            const int k = k0 + 16 * st;
            const bool in = k + 4 * q < k1;   // false past the split's end: zeros on both sides
#pragma unroll
            for (int m = 0; m < MR; ++m) cv[m] = buf_ld128(rc, in ? coff[m] + static_cast<uint32_t>(k) * 4u : kBufOOB);
            const uint32_t kq = static_cast<uint32_t>(k) * pp * 4u;   // bytes of row quad k / 4
#pragma unroll
            for (int b = 0; b < NB; ++b) qv[b] = buf_ld128(rq, in ? kq + qoff + 256u * b : kBufOOB);
        };
        const int iters = ((nsteps - wave + 3) / 4 + ST - 1) / ST;
        u32x4 cv[ST][MR], qv[ST][NB];
        int s = wave;
#pragma unroll
        for (int i = 0; i < ST - 1; ++i) load(s + 4 * i, cv[i], qv[i]);
        for (int it = 0; it < iters; ++it) {
#pragma unroll
            for (int i = 0; i < ST; ++i) {
                load(s + 4 * (i + ST - 1), cv[(i + ST - 1) % ST], qv[(i + ST - 1) % ST]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int m = 0; m < MR; ++m)
#pragma unroll
                        for (int b = 0; b < NB; ++b)
                            acc[m][b] = mfma16_f32(__uint_as_float(cv[i][m][e]), __uint_as_float(qv[i][b][e]),
                                                   acc[m][b]);
            }
            s += 4 * ST;
        }
    }
    cq_fold_store<NB, MR>(acc, fold, lane, wave, m0, n4, Zs);
}

// Z = sum of the splits' partials, in split order (128-bit elements).
__global__ __launch_bounds__(256) void k_cq_sum(const f32x4 *__restrict__ Zs, int64_t n_vec, int splits,
                                                f32x4 *__restrict__ Z) {
    const int64_t v = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (v >= n_vec) return;
    f32x4 s = Zs[v];
    for (int t = 1; t < splits; ++t) s += Zs[static_cast<size_t>(t) * n_vec + v];
    Z[v] = s;
}

// Partial Gram sums G_c[a][b] = sum over rows r of chunk c of X[r][a] Y[r][b]
// (fp64), a, b < p, for X, Y in row quads (n4 rows, zero past n), one
// workgroup per chunk of kGramRows rows (64: 224 workgroups at n = 14336).
// Rows are staged through LDS kGramChunk at a time (a longer chunk loads the
// next rows into registers while the current ones are summed); an LDS read
// of 128 bits gives one column's values in four consecutive rows.  PMAX (32,
// 64 or 128) bounds p; a workgroup forms at most 4096 of the p x p sums (16
// per thread), the blockIdx.y-th group of them.
template <int PMAX>
__global__ __launch_bounds__(256) void k_gram_part(const float *__restrict__ X, const float *__restrict__ Y, int n,
                                                   int p, int pp, double *__restrict__ part) {
    constexpr int kV = PMAX / 16;               // 128-bit loads per thread and operand, at most
    constexpr int kU = PMAX * PMAX / 256 < 16 ? PMAX * PMAX / 256 : 16;   // outputs per thread, at most
    __shared__ f32x4 xs[kGramChunk / 4 * PMAX], ys[kGramChunk / 4 * PMAX];
    const int tid = threadIdx.x;
    const int n4 = round4(n);
    const int r0 = blockIdx.x * kGramRows;
    const int rend = min(n4, r0 + kGramRows);
    const int np = p * p;
    const int nv = pp / 16;                     // 128-bit loads per thread of a full chunk
    const f32x4 *X4 = reinterpret_cast<const f32x4 *>(X);
    const f32x4 *Y4 = reinterpret_cast<const f32x4 *>(Y);
    f32x4 xr[kV], yr[kV];
    auto fetch = [&](int c0) {
        const int lim = (min(kGramChunk, rend - c0) / 4) * pp;   // 128-bit elements of this chunk
        const size_t base = static_cast<size_t>(c0 / 4) * pp;
#pragma unroll
        for (int v = 0; v < kV; ++v) {
            const int f = tid + 256 * v;
            const bool ok = v < nv && f < lim;
            xr[v] = ok ? X4[base + f] : f32x4{0.f, 0.f, 0.f, 0.f};
            yr[v] = ok ? Y4[base + f] : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };
    double acc[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) acc[u] = 0.0;
    const int e0 = blockIdx.y * 256 * kU;       // first output of this workgroup
    if (r0 < rend) fetch(r0);
    for (int c0 = r0; c0 < rend; c0 += kGramChunk) {
        const int nq = min(kGramChunk, rend - c0) / 4;
#pragma unroll
        for (int v = 0; v < kV; ++v) {
            const int f = tid + 256 * v;
            if (v < nv && f < nq * pp) {
                xs[f] = xr[v];
                ys[f] = yr[v];
            }
        }
        __syncthreads();
        if (c0 + kGramChunk < rend) fetch(c0 + kGramChunk);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int e = e0 + tid + 256 * u;
            if (e < np) {
                const int a = e / p, b = e - (e / p) * p;
                double s = acc[u];
                for (int qq = 0; qq < nq; ++qq) {
                    const f32x4 xv = xs[qq * pp + a], yv = ys[qq * pp + b];
#pragma unroll
                    for (int r = 0; r < 4; ++r) s = fma(static_cast<double>(xv[r]), static_cast<double>(yv[r]), s);
                }
                acc[u] = s;
            }
        }
        __syncthreads();
    }
    double *dst = part + static_cast<size_t>(blockIdx.x) * np;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const int e = e0 + tid + 256 * u;
        if (e < np) dst[e] = acc[u];
    }
}

void launch_gram(const float *X, const float *Y, int n, int p, int pp, double *part, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((round4(n) + kGramRows - 1) / kGramRows),
                    static_cast<unsigned>((p * p + 4095) / 4096));
    if (pp <= 32) hipLaunchKernelGGL(k_gram_part<32>, grid, dim3(256), 0, s, X, Y, n, p, pp, part);
    else if (pp <= 64) hipLaunchKernelGGL(k_gram_part<64>, grid, dim3(256), 0, s, X, Y, n, p, pp, part);
    else hipLaunchKernelGGL(k_gram_part<128>, grid, dim3(256), 0, s, X, Y, n, p, pp, part);
}

// G = sum of the chunk partials, in chunk order, into A (all threads).  The
// partials were just written by CUs all over the chip and this workgroup
// runs alone, so the sum is bound by memory latency: a thread sums four
// elements at a time with eight chunks of each in flight (32 loads).
__device__ __forceinline__ void sum_partials(const double *__restrict__ part, int chunks, int np, double *A,
                                             int tid) {
    for (int e0 = tid; e0 < np; e0 += 4 * 256) {
        double s[4] = {0.0, 0.0, 0.0, 0.0};
        int c = 0;
        for (; c + 8 <= chunks; c += 8) {
            double v[4][8];
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int w = 0; w < 8; ++w)
                    v[u][w] = e0 + 256 * u < np ? part[static_cast<size_t>(c + w) * np + e0 + 256 * u] : 0.0;
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int w = 0; w < 8; ++w) s[u] += v[u][w];
        }
        for (; c < chunks; ++c)
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (e0 + 256 * u < np) s[u] += part[static_cast<size_t>(c) * np + e0 + 256 * u];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (e0 + 256 * u < np) A[e0 + 256 * u] = s[u];
    }
}

// G = the sum of the chunk partials, written over chunk 0's slot.  The Gram
// partials come in 64-row chunks (224 at n = 14336: 1.8 MB at p = 32, 29 MB
// at p = 128), too many for one workgroup to gather; spread over the chip
// they take a few microseconds, and the one-workgroup kernels then read a
// single chunk.  A workgroup takes 64 elements; wave w sums the w-th quarter
// of the chunks of each, in chunk order, and the quarters are added in a
// fixed order, ((q0 + q1) + q2) + q3, after every chunk has been read.
__global__ __launch_bounds__(256) void k_sum_parts(double *__restrict__ part, int chunks, int np) {
    __shared__ double q[4][kWave];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int e = blockIdx.x * kWave + lane;
    const int per = (chunks + 3) / 4;
    const int c0 = min(chunks, w * per), c1 = min(chunks, c0 + per);
    double s = 0.0;
    if (e < np) {
        int c = c0;
        for (; c + 8 <= c1; c += 8) {
            double v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = part[static_cast<size_t>(c + u) * np + e];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; c < c1; ++c) s += part[static_cast<size_t>(c) * np + e];
    }
    q[w][lane] = s;
    __syncthreads();
    if (w == 0 && e < np) part[e] = ((q[0][lane] + q[1][lane]) + q[2][lane]) + q[3][lane];
}

// f(std::integral_constant<int, I>{}) for I = 0 .. N - 1, expanded by the
// front end: a register array indexed by I stays in registers however long
// the body is (the loop unroller gives up on long bodies).
template <typename F, int... I>
__device__ __forceinline__ void static_for_seq(F &f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// a[i] -= v[i] f for i < RPT, v RPT consecutive doubles in LDS (16-byte
// aligned): read 16 at a time, one group ahead of its FMAs, so that at most
// two groups are live next to a; a is in registers on return.
template <int RPT>
__device__ __forceinline__ void axpy_lds(double (&a)[RPT], const double *v, double f) {
    static_assert(RPT % 16 == 0, "groups of 16");
    constexpr int G = RPT / 16;
    const double2 *v2 = reinterpret_cast<const double2 *>(v);
    double2 cur[8], nxt[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) cur[k] = v2[k];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        if (g + 1 < G) {
#pragma unroll
            for (int k = 0; k < 8; ++k) nxt[k] = v2[8 * (g + 1) + k];
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            a[16 * g + 2 * k] = fma(-cur[k].x, f, a[16 * g + 2 * k]);
            a[16 * g + 2 * k + 1] = fma(-cur[k].y, f, a[16 * g + 2 * k + 1]);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < 8; ++k) cur[k] = nxt[k];
    }
    // the updated values are materialised here: left to itself the compiler
    // sinks each step's FMAs towards the step that reads the row, keeping
    // every loaded value live until then
#pragma unroll
    for (int i = 0; i < RPT; ++i) asm volatile("" : "+v"(a[i]));
}

// One workgroup; the matrix is padded to PM (32, 64 or 128) with the
// identity, whose factor and inverse are the identity.  Thread (c, h) keeps
// rows RPT h .. RPT h + RPT - 1 of column c in registers (RPT = min(PM, 64)):
// for PM <= 64 one wave, lane c holding the whole column; for PM = 128 four
// waves, c = 64 (wave & 1) + lane and h = wave >> 1.  The shifted Cholesky
// G + eps (tr G / p) I = R^T R runs in outer-product form: step j passes row
// j through LDS (zeros left of the diagonal) and every thread updates its
// entries below it, A_rc -= A_jr (A_jc / A_jj); each step is the same RPT
// FMAs in every thread, the zeros leaving the rows above it unchanged.  Row
// r of R is then row r of the updated matrix over sqrt(A_rr) (a non-positive
// pivot, which cannot follow the shift, is taken as 1).  X = R^{-1} solves
// R X = I by back substitution in the same form with R in LDS: steps
// j = PM - 1 .. 0 finish row j of X, X_jc = B_jc / R_jj, pass it through LDS
// and update the rows above it, B_rc -= R_rj X_jc.  With four waves a
// barrier follows each step's row (two row buffers alternate); one wave
// needs none, its LDS operations taking effect in program order.  All fp64.
// Writes R^{-T} [p][p] (R^{-1} transposed: zero above the diagonal),
// through LDS so that the stores are coalesced.
template <int PM>
__global__ __launch_bounds__(256) void k_chol_inv_cols(const double *__restrict__ part, int chunks, int p,
                                                       double *__restrict__ RinvT) {
    constexpr int RPT = PM < 64 ? PM : 64;
    constexpr int NW = PM <= 64 ? 1 : 4;   // waves that factorise
    constexpr int RS = PM + 2;   // stride of the column-major copies of R and R^{-T} (even: 16-byte pairs)
    __shared__ __attribute__((aligned(16))) double A[PM * RS];   // G [p][p]; then R by columns; then R^{-T} by rows
    __shared__ __attribute__((aligned(16))) double buf[2][PM];
    __shared__ double rdiag[PM];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = NW == 4 ? 64 * (wave & 1) + lane : lane;
    const int h = NW == 4 ? wave >> 1 : 0;
    const bool col = c < PM;   // lanes past PM (PM = 32) hold no column
    sum_partials(part, chunks, p * p, A, tid);
    __syncthreads();
    if (wave >= NW) return;
    auto sync = [] {
        if constexpr (NW > 1) __syncthreads();
    };
    double tr = 0.0;
    for (int r = 0; r < p; ++r) tr += A[r * p + r];   // the same order in every thread
    const double shift = 1e-12 * (tr > 0.0 ? tr / p : 1.0);
    double a[RPT];
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
        const int r = RPT * h + i;
        const double g = A[min(r, p - 1) * p + min(c, p - 1)];   // clamped: padding is selected below
        a[i] = r < p && c < p ? (r == c ? g + shift : g) : r == c ? 1.0 : 0.0;
    }
    if constexpr (NW > 1) __syncthreads();   // G is overwritten below
    else __builtin_amdgcn_wave_barrier();
    static_for<PM>([&](auto step) __attribute__((always_inline)) {
        constexpr int j = decltype(step)::value;
        constexpr int hj = j / RPT, jj = j % RPT;
        double *row = buf[j & 1];
        if (h == hj && col) row[c] = c >= j ? a[jj] : 0.0;   // zeros left of the diagonal: no update there
        sync();
        // one wave: the pivot from lane j's register and f from the lane's own
        // (the values the row holds), so the reciprocal need not wait for LDS
        const double d = NW == 1 ? readlane_d(a[jj], j) : row[j];
        const double e = d > 0.0 ? d : 1.0;
        if (tid == 0) rdiag[j] = e;
        const double f = col && c > j ? (NW == 1 ? a[jj] : row[c]) / e : 0.0;
        const double keep = a[jj];   // row j itself is final
        axpy_lds<RPT>(a, row + RPT * h, f);
        a[jj] = h == hj ? keep : a[jj];
    });
    sync();   // the pivots are complete
    if (tid < PM) rdiag[tid] = sqrt(rdiag[tid]);   // R_rr
    sync();
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
        const int r = RPT * h + i;
        const double rr = rdiag[r];
        if (col) A[c * RS + r] = r < c ? a[i] / rr : r == c ? rr : 0.0;   // R_rc, column c contiguous
        a[i] = r == c ? 1.0 : 0.0;
    }
    sync();
    static_for<PM>([&](auto step) __attribute__((always_inline)) {
        constexpr int j = PM - 1 - decltype(step)::value;
        constexpr int hj = j / RPT, jj = j % RPT;
        double *row = buf[j & 1];
        const double *Rj = A + j * RS;   // column j of R
        if (h == hj) {
            a[jj] = a[jj] / Rj[j];
            if (NW > 1 && col) row[c] = a[jj];
        }
        sync();
        // one wave: row j of X is the lane's own register
        const double x = col ? (NW == 1 ? a[jj] : row[c]) : 0.0;
        const double keep = a[jj];   // row j of X is final; R is zero below its diagonal
        axpy_lds<RPT>(a, Rj + RPT * h, x);
        a[jj] = h == hj ? keep : a[jj];
    });
    sync();   // every read of R is done
    if (col) {
#pragma unroll
        for (int i = 0; i < RPT; ++i) A[c * RS + RPT * h + i] = a[i];   // row c of R^{-T} is column c of R^{-1}
    }
    sync();
    for (int e = tid; e < p * p; e += kWave * NW) {
        const int r = e / p;
        RinvT[e] = A[r * RS + (e - r * p)];
    }
}

void launch_chol_inv(const double *part, int chunks, int p, double *RinvT, hipStream_t s) {
    if (p <= 32) hipLaunchKernelGGL(k_chol_inv_cols<32>, dim3(1), dim3(256), 0, s, part, chunks, p, RinvT);
    else if (p <= 64) hipLaunchKernelGGL(k_chol_inv_cols<64>, dim3(1), dim3(256), 0, s, part, chunks, p, RinvT);
    else hipLaunchKernelGGL(k_chol_inv_cols<kMaxP>, dim3(1), dim3(256), 0, s, part, chunks, p, RinvT);
}

// Q = Z R^{-1} in row quads.  Lane = one row quad, wave = four consecutive
// columns j0 .. j0 + 3: entry (i, j) = sum over m <= j of Z[i][m]
// R^{-1}[m][j] in fp64 (fp32 result), m ascending.  R^{-1} comes transposed
// (column j a contiguous row, zero past the diagonal), so the four columns
// share one loop to j0 + 3, the entries past a column's diagonal adding exact
// zeros; its entries are the same across the wave (scalar loads), and each
// 128-bit load of Z feeds 16 FMAs.  The padding columns j >= p are zero.
__global__ __launch_bounds__(256) void k_apply_rinv(const float *__restrict__ Z, int n, int p, int pp,
                                                    const double *__restrict__ RinvT, float *__restrict__ Q) {
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    const int j0 = 4 * (4 * static_cast<int>(blockIdx.y) + wave);
    const int64_t nq = round4(n) / 4;
    const int64_t quad = static_cast<int64_t>(blockIdx.x) * kWave + lane;
    const bool qin = quad < nq;
    double acc[4][4];   // [column j0 + u][row 4 quad + r]
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[u][r] = 0.0;
    if (j0 < p) {
        const f32x4 *Z4 = reinterpret_cast<const f32x4 *>(Z) + (qin ? quad : 0) * pp;
        const int mend = min(j0 + 4, p);
        const double *R[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) R[u] = RinvT + static_cast<size_t>(min(j0 + u, p - 1)) * p;
#pragma unroll 4
        for (int m = 0; m < mend; ++m) {
            const f32x4 z = Z4[m];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const double rv = j0 + u < p ? R[u][m] : 0.0;
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[u][r] = fma(static_cast<double>(z[r]), rv, acc[u][r]);
            }
        }
    }
    if (!qin) return;
    f32x4 *Q4 = reinterpret_cast<f32x4 *>(Q) + quad * pp + j0;
#pragma unroll
    for (int u = 0; u < 4; ++u)
        Q4[u] = f32x4{static_cast<float>(acc[u][0]), static_cast<float>(acc[u][1]), static_cast<float>(acc[u][2]),
                      static_cast<float>(acc[u][3])};
}

// One workgroup: T = (sum of the chunk partials of Q^T Z), symmetrised, is
// diagonalised by round-robin parallel cyclic Jacobi in fp64.  Each round
// applies m/2 disjoint plane rotations (m = p rounded up to even; a pair
// with the padding index p is the identity), each zeroing T[a][b] (the
// symmetric 2 x 2 Schur decomposition).  A round's pairs partition the
// indices, so the block of T on the rows of pair P and the columns of pair
// Q becomes G_P T_PQ G_Q^T with G = [[c, -s], [s, c]]: the same products as
// rotating the rows and then the columns, formed by one thread per block in
// place, two barriers per round.  Sweeps stop when the off-diagonal mass is
// below 1e-30 of the total, or after kJacobiSweeps.  The eigenvectors are
// not formed here: each round's (c, s) go to `rot` [round][m/2] and the
// number of rounds to *rounds, and k_jacobi_replay applies them to W^T.
// Writes theta [p].  T stays in LDS (PM = 64 or 128).
template <int PM>
__global__ __launch_bounds__(256) void k_jacobi_rot(const double *__restrict__ part, int chunks, int p,
                                                    double2 *__restrict__ rot, int *__restrict__ rounds,
                                                    double *__restrict__ theta) {
    __shared__ double T[PM * PM];
    __shared__ double cs[PM / 2], sn[PM / 2];
    __shared__ int pa[PM / 2], pb[PM / 2];
    __shared__ double red[8];
    const int tid = threadIdx.x, np = p * p, lane = tid & 63, wave = tid >> 6;
    sum_partials(part, chunks, np, T, tid);
    __syncthreads();
    for (int e = tid; e < np; e += 256) {
        const int a = e / p, b = e - (e / p) * p;
        if (a < b) {
            const double v = 0.5 * (T[a * p + b] + T[b * p + a]);
            T[a * p + b] = v;
            T[b * p + a] = v;
        }
    }
    __syncthreads();
    const int m = p + (p & 1);   // players of the round-robin schedule
    const int half = m / 2;
    int done = 0;   // rounds applied
    for (int sweep = 0; sweep < kJacobiSweeps; ++sweep) {
        double off = 0.0, all = 0.0;
        for (int e = tid; e < np; e += 256) {
            const int a = e / p, b = e - (e / p) * p;
            const double v = T[e] * T[e];
            all += v;
            if (a != b) off += v;
        }
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            off += __shfl_xor(off, o, kWave);
            all += __shfl_xor(all, o, kWave);
        }
        if (lane == 0) {
            red[2 * wave] = off;
            red[2 * wave + 1] = all;
        }
        __syncthreads();
        const double off_sum = ((red[0] + red[2]) + red[4]) + red[6];
        const double all_sum = ((red[1] + red[3]) + red[5]) + red[7];
        if (!(off_sum > 1e-30 * all_sum)) break;   // uniform: every thread read the same sums
        for (int rnd = 0; rnd < m - 1; ++rnd, ++done) {   // red is rewritten only after this round's barriers
            if (tid < half) {
                // circle method: position 0 fixed, positions 1 .. m - 1 turn by one each round
                auto player = [&](int pos) { return pos == 0 ? 0 : 1 + (pos - 1 + rnd) % (m - 1); };
                int a = player(tid), b = player(m - 1 - tid);
                if (a > b) {
                    const int t = a;
                    a = b;
                    b = t;
                }
                double c = 1.0, sv = 0.0;
                if (b < p) {
                    const double apq = T[a * p + b];
                    if (apq != 0.0) {
                        const double tau = (T[b * p + b] - T[a * p + a]) / (2.0 * apq);
                        const double t = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
                        c = 1.0 / sqrt(1.0 + t * t);
                        sv = t * c;
                    }
                }
                pa[tid] = a;
                pb[tid] = b;
                cs[tid] = c;
                sn[tid] = sv;
                rot[static_cast<size_t>(done) * half + tid] = double2{c, sv};
            }
            __syncthreads();
            for (int e = tid; e < half * half; e += 256) {
                const int P = e / half, Q = e - (e / half) * half;
                const int a = pa[P], b = pb[P], c2 = pa[Q], d = pb[Q];
                const bool bp = b < p, bq = d < p;
                const double cp = cs[P], sp = sn[P], cq = cs[Q], sq = sn[Q];
                const double t00 = T[a * p + c2], t01 = bq ? T[a * p + d] : 0.0;
                const double t10 = bp ? T[b * p + c2] : 0.0, t11 = bp && bq ? T[b * p + d] : 0.0;
                const double u00 = cp * t00 - sp * t10, u01 = cp * t01 - sp * t11;
                const double u10 = sp * t00 + cp * t10, u11 = sp * t01 + cp * t11;
                T[a * p + c2] = cq * u00 - sq * u01;
                if (bq) T[a * p + d] = sq * u00 + cq * u01;
                if (bp) T[b * p + c2] = cq * u10 - sq * u11;
                if (bp && bq) T[b * p + d] = sq * u10 + cq * u11;
            }
            __syncthreads();
        }
    }
    if (tid == 0) *rounds = done;
    for (int a = tid; a < p; a += 256) theta[a] = T[a * p + a];
}

// W^T (rows: the eigenvectors of T) = the product of the logged rotations
// applied to the identity.  A rotation of pair (a, b) turns rows a and b of
// W^T, so every column evolves on its own: workgroup i (one wave) keeps
// column i in LDS and takes the rounds in order, lane q turning entries a, b
// of the round's pair q by its (c, s), with the pairs found by the same
// circle method.  The LDS operations of one wave take effect in program
// order, so a round reads what the one before it wrote.  The rotations'
// (c, s) are loaded eight rounds ahead.  Writes Wt [p][p].
__global__ __launch_bounds__(64) void k_jacobi_replay(const double2 *__restrict__ rot, const int *__restrict__ rounds,
                                                      int p, double *__restrict__ Wt) {
    constexpr int kAhead = 8;
    __shared__ double col[kMaxP];
    const int i = blockIdx.x, lane = threadIdx.x;
    for (int a = lane; a < p; a += kWave) col[a] = a == i ? 1.0 : 0.0;
    const int m = p + (p & 1), half = m / 2;
    const int nr = *rounds;
    const bool active = lane < half;
    // circle positions of this lane's pair, advanced by one (mod m - 1) each round
    int ta = lane == 0 ? -1 : lane - 1;        // -1: the fixed position 0
    int tb = m - 1 - lane - 1;
    double2 g[kAhead], gn[kAhead];
#pragma unroll
    for (int u = 0; u < kAhead; ++u)
        g[u] = active && u < nr ? rot[static_cast<size_t>(u) * half + lane] : double2{1.0, 0.0};
    for (int r0 = 0; r0 < nr; r0 += kAhead) {
#pragma unroll
        for (int u = 0; u < kAhead; ++u) {
            const int r = r0 + kAhead + u;
            gn[u] = active && r < nr ? rot[static_cast<size_t>(r) * half + lane] : double2{1.0, 0.0};
        }
#pragma unroll
        for (int u = 0; u < kAhead; ++u) {
            if (r0 + u < nr && active) {
                int a = ta < 0 ? 0 : 1 + ta, b = 1 + tb;
                if (a > b) {
                    const int t = a;
                    a = b;
                    b = t;
                }
                if (b < p) {
                    const double c = g[u].x, sv = g[u].y;
                    const double wa = col[a], wb = col[b];
                    col[a] = c * wa - sv * wb;
                    col[b] = sv * wa + c * wb;
                }
            }
            ta = ta < 0 ? ta : ta + 1 == m - 1 ? 0 : ta + 1;
            tb = tb + 1 == m - 1 ? 0 : tb + 1;
        }
#pragma unroll
        for (int u = 0; u < kAhead; ++u) g[u] = gn[u];
    }
    for (int a = lane; a < p; a += kWave) Wt[static_cast<size_t>(a) * p + i] = col[a];
}

// Ritz vectors of the k largest theta (decreasing; equal values in index
// order): V[e][i] = sum_j Q[i][j] Wt[order_e][j] (fp64 sums in j order, fp32
// result; Q in row quads), and eigvals[e].  Workgroup (x, y) forms Ritz
// vectors kRitzE y .. kRitzE y + kRitzE - 1 on 1024 rows: a thread takes one
// row quad, one 128-bit load of Q per j feeding 4 kRitzE fp64 FMAs, with the
// selected rows of Wt in LDS.  Each theta's rank is counted by its own
// thread.
constexpr int kRitzE = 16;
__global__ __launch_bounds__(256) void k_ritz(const float *__restrict__ Q, int n, int p, int pp, int k,
                                              const double *__restrict__ Wt, const double *__restrict__ theta,
                                              float *__restrict__ V, float *__restrict__ eigvals) {
    __shared__ double th[kMaxP];
    __shared__ int order[kRitzE];
    __shared__ double w[kRitzE * kMaxP];
    const int tid = threadIdx.x, e0 = blockIdx.y * kRitzE;
    const int ne = min(kRitzE, k - e0);
    for (int a = tid; a < p; a += 256) th[a] = theta[a];
    __syncthreads();
    for (int a = tid; a < p; a += 256) {
        int rank = 0;   // larger first, lower index first among equals
        for (int b = 0; b < p; ++b) rank += th[b] > th[a] || (th[b] == th[a] && b < a);
        if (rank >= e0 && rank < e0 + ne) order[rank - e0] = a;
    }
    __syncthreads();
    for (int x = tid; x < kRitzE * p; x += 256) {
        const int e = x / p, j = x - (x / p) * p;
        w[e * kMaxP + j] = e < ne ? Wt[static_cast<size_t>(order[e]) * p + j] : 0.0;
    }
    if (blockIdx.x == 0 && tid < ne && eigvals) eigvals[e0 + tid] = static_cast<float>(th[order[tid]]);
    __syncthreads();
    const int quad = blockIdx.x * 256 + tid;   // rows 4 quad .. 4 quad + 3
    if (4 * quad >= n) return;
    const f32x4 *Q4 = reinterpret_cast<const f32x4 *>(Q) + static_cast<size_t>(quad) * pp;
    double acc[4][kRitzE];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int e = 0; e < kRitzE; ++e) acc[r][e] = 0.0;
    for (int j = 0; j < p; ++j) {
        const f32x4 q = Q4[j];
#pragma unroll
        for (int e = 0; e < kRitzE; ++e) {
            const double we = w[e * kMaxP + j];
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[r][e] = fma(static_cast<double>(q[r]), we, acc[r][e]);
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = 4 * quad + r;
        if (i >= n) break;
#pragma unroll
        for (int e = 0; e < kRitzE; ++e)
            if (e < ne) V[static_cast<size_t>(e0 + e) * n + i] = static_cast<float>(acc[r][e]);
    }
}

// One workgroup per Ritz vector: the index of its largest magnitude (lowest
// index among equal magnitudes) sets the sign; the row of P is written in the
// output dtype.
template <typename TOut>
__global__ __launch_bounds__(256) void k_pca_out(const float *__restrict__ V, int n, TOut *__restrict__ P,
                                                 int64_t ld_p) {
    __shared__ float bv[256];
    __shared__ int bi[256];
    const int e = blockIdx.x, tid = threadIdx.x;
    const float *v = V + static_cast<size_t>(e) * n;
    float best = -1.f;
    int idx = 0x7fffffff;
    for (int i = tid; i < n; i += 256) {
        const float a = fabsf(v[i]);
        if (a > best) {   // increasing i: the first of equal magnitudes is kept
            best = a;
            idx = i;
        }
    }
    bv[tid] = best;
    bi[tid] = idx;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (tid < w) {
            const float ob = bv[tid + w];
            const int oi = bi[tid + w];
            if (ob > bv[tid] || (ob == bv[tid] && oi < bi[tid])) {
                bv[tid] = ob;
                bi[tid] = oi;
            }
        }
        __syncthreads();
    }
    const float sgn = v[bi[0]] < 0.f ? -1.f : 1.f;
    for (int i = tid; i < n; i += 256) store_out<TOut>(P + static_cast<int64_t>(e) * ld_p + i, sgn * v[i]);
}

}  // namespace

size_t act_cov_ws_bytes(int B, int T) {
    const size_t slabs = static_cast<size_t>(B) * ((T + ST - 1) / ST);
    return align256(sizeof(int) * slabs) + align256(sizeof(uint32_t) * slabs) + 256;
}

hipError_t launch_act_cov_group(const void *const *a, float *const *C, const int *n, int count, bool bf16, int B,
                                int T, const uint8_t *mask, void *ws, hipStream_t s) {
    if (B == 0 || T == 0 || count == 0) return hipSuccess;
    if (count < 0 || count > kMaxActCovGroup) return hipErrorInvalidValue;
    const int spe = (T + ST - 1) / ST;
    const size_t slabs = static_cast<size_t>(B) * spe;
    char *w = static_cast<char *>(ws);
    int *list = reinterpret_cast<int *>(w);
    uint32_t *bits = reinterpret_cast<uint32_t *>(w + align256(sizeof(int) * slabs));
    int *n_slabs = reinterpret_cast<int *>(w + align256(sizeof(int) * slabs) + align256(sizeof(uint32_t) * slabs));
    hipLaunchKernelGGL(k_slab_prep, dim3(1), dim3(1024), 0, s, mask, B, T, spe, list, bits, n_slabs);
    if (bf16) {
        // the largest factors first, so that the small ones fill the last rounds
        int order[kMaxActCovGroup];
        for (int i = 0; i < count; ++i) order[i] = i;
        std::stable_sort(order, order + count, [&](int x, int y) { return n[x] > n[y]; });
        ActCovArgs g;
        g.count = count;
        int64_t slots = 0;
        for (int i = 0; i < count; ++i) {
            const int f = order[i];
            const int nt = (n[f] + CT - 1) / CT;
            slots += tile_slots(nt);
            if (slots > INT32_MAX) return hipErrorInvalidValue;
            g.f[i] = {static_cast<const bf16_bits *>(a[f]), C[f], n[f], nt, static_cast<int>(slots)};
        }
        hipLaunchKernelGGL(k_act_cov_dma, dim3(static_cast<unsigned>(slots)), dim3(256), 0, s, g, T, spe, list,
                           bits, n_slabs);
    } else {
        for (int f = 0; f < count; ++f) {
            const unsigned nb = static_cast<unsigned>((n[f] + 15) / 16);
            hipLaunchKernelGGL(k_act_cov_f32, dim3(nb, nb), dim3(256), 0, s, static_cast<const float *>(a[f]), T,
                               n[f], spe, list, bits, n_slabs, C[f]);
        }
    }
    return hipGetLastError();
}

hipError_t launch_act_cov(const void *a, bool bf16, int B, int T, int n, const uint8_t *mask, float *C, void *ws,
                          hipStream_t s) {
    return launch_act_cov_group(&a, &C, &n, 1, bf16, B, T, mask, ws, s);
}

}  // namespace logra

namespace logra {
namespace {

struct PcaLayout {
    float *Q, *Z, *Zs;
    double *part, *RinvT, *Wt, *theta;
    double2 *rot;   // the Jacobi rotations, [round][m/2]
    int *rounds;
};

inline int pca_p(int n, int k) {
    const int w = 2 * k > 16 ? 2 * k : 16;   // at least one MFMA column block of vectors
    return w < n ? w : n;
}
inline int pca_pp(int n, int k) { return (pca_p(n, k) + 15) / 16 * 16; }
inline int gram_chunks(int n) { return (round4(n) + kGramRows - 1) / kGramRows; }
inline size_t block_floats(int n, int pp) { return static_cast<size_t>(round4(n)) * pp; }
inline size_t rot_bytes(int p) {
    const int m = p + (p & 1);
    return sizeof(double2) * static_cast<size_t>(kJacobiSweeps) * (m - 1) * (m / 2);
}

// Z = C Q: row blocks of 16 MR rows per workgroup, and the columns of C cut
// into splits of kr (a multiple of 64, at least 512 unless n is smaller) so
// that the grid has about 2048 workgroups.
inline int cq_mr(int pp) { return pp / 16 <= 4 ? 4 : 2; }
inline int cq_kr(int n, int pp) {
    const int rb = (n + 16 * cq_mr(pp) - 1) / (16 * cq_mr(pp));
    int sp = (2048 + rb - 1) / rb;
    sp = sp < n / 512 ? sp : n / 512;
    sp = sp > 1 ? sp : 1;
    return ((n + sp - 1) / sp + 63) / 64 * 64;
}
inline int cq_splits(int n, int pp) { return (n + cq_kr(n, pp) - 1) / cq_kr(n, pp); }

PcaLayout pca_layout(void *ws, int n, int k) {
    const int p = pca_p(n, k), pp = pca_pp(n, k);
    char *w = static_cast<char *>(ws);
    PcaLayout L;
    L.Q = reinterpret_cast<float *>(w);
    w += align256(sizeof(float) * block_floats(n, pp));
    L.Z = reinterpret_cast<float *>(w);
    w += align256(sizeof(float) * block_floats(n, pp));
    const int sp = cq_splits(n, pp);
    L.Zs = sp > 1 ? reinterpret_cast<float *>(w) : L.Z;
    w += sp > 1 ? align256(sizeof(float) * block_floats(n, pp) * sp) : 0;
    L.part = reinterpret_cast<double *>(w);
    w += align256(sizeof(double) * static_cast<size_t>(gram_chunks(n)) * p * p);
    L.RinvT = reinterpret_cast<double *>(w);
    w += align256(sizeof(double) * static_cast<size_t>(p) * p);
    L.Wt = reinterpret_cast<double *>(w);
    w += align256(sizeof(double) * static_cast<size_t>(p) * p);
    L.theta = reinterpret_cast<double *>(w);
    w += align256(sizeof(double) * p);
    L.rot = reinterpret_cast<double2 *>(w);
    w += align256(rot_bytes(p));
    L.rounds = reinterpret_cast<int *>(w);
    return L;
}

template <int NB>
void launch_cq_nb(const float *C, int n, const float *Q, float *Zs, hipStream_t s) {
    constexpr int MR = NB <= 4 ? 4 : 2;
    const int kr = cq_kr(n, 16 * NB);
    const dim3 grid(static_cast<unsigned>((n + 16 * MR - 1) / (16 * MR)), static_cast<unsigned>((n + kr - 1) / kr));
    if constexpr (NB <= 4)
        hipLaunchKernelGGL((k_cq_dma<NB, MR>), grid, dim3(256), 0, s, C, n, Q, kr, Zs);
    else
        hipLaunchKernelGGL((k_cq_regs<NB, MR>), grid, dim3(256), 0, s, C, n, Q, kr, Zs);
}

hipError_t launch_cq(const PcaLayout &L, const float *C, int n, int pp, const float *Q, float *Z, hipStream_t s) {
    const int sp = cq_splits(n, pp);
    float *dst = sp > 1 ? L.Zs : Z;
    switch (pp / 16) {
        case 1: launch_cq_nb<1>(C, n, Q, dst, s); break;
        case 2: launch_cq_nb<2>(C, n, Q, dst, s); break;
        case 3: launch_cq_nb<3>(C, n, Q, dst, s); break;
        case 4: launch_cq_nb<4>(C, n, Q, dst, s); break;
        case 5: launch_cq_nb<5>(C, n, Q, dst, s); break;
        case 6: launch_cq_nb<6>(C, n, Q, dst, s); break;
        case 7: launch_cq_nb<7>(C, n, Q, dst, s); break;
        default: launch_cq_nb<8>(C, n, Q, dst, s); break;
    }
    if (sp > 1) {
        const int64_t nv = static_cast<int64_t>(block_floats(n, pp) / 4);
        hipLaunchKernelGGL(k_cq_sum, dim3(static_cast<unsigned>((nv + 255) / 256)), dim3(256), 0, s,
                           reinterpret_cast<const f32x4 *>(L.Zs), nv, sp, reinterpret_cast<f32x4 *>(Z));
    }
    return hipGetLastError();
}

// Sums the Gram partials on the chip; returns the chunk count left for the
// one-workgroup kernel that follows.
int sum_parts(double *part, int chunks, int p, hipStream_t s) {
    if (chunks == 1) return chunks;
    hipLaunchKernelGGL(k_sum_parts, dim3(static_cast<unsigned>((p * p + kWave - 1) / kWave)), dim3(256), 0, s, part,
                       chunks, p * p);
    return 1;
}

// Q = orthonormalised Z (shifted CholQR)
void cholqr(const PcaLayout &L, int n, int p, int pp, const float *Z, float *Q, hipStream_t s) {
    launch_gram(Z, Z, n, p, pp, L.part, s);
    launch_chol_inv(L.part, sum_parts(L.part, gram_chunks(n), p, s), p, L.RinvT, s);
    const dim3 grid(static_cast<unsigned>((round4(n) / 4 + kWave - 1) / kWave), static_cast<unsigned>(pp / 16));
    hipLaunchKernelGGL(k_apply_rinv, grid, dim3(256), 0, s, Z, n, p, pp, L.RinvT, Q);
}

}  // namespace

size_t pca_ws_bytes(int n, int k) {
    const int p = pca_p(n, k), pp = pca_pp(n, k);
    const int sp = cq_splits(n, pp);
    return 2 * align256(sizeof(float) * block_floats(n, pp)) +
           (sp > 1 ? align256(sizeof(float) * block_floats(n, pp) * sp) : 0) +
           align256(sizeof(double) * static_cast<size_t>(gram_chunks(n)) * p * p) +
           2 * align256(sizeof(double) * static_cast<size_t>(p) * p) + align256(sizeof(double) * p) +
           align256(rot_bytes(p)) + align256(sizeof(int));
}

hipError_t launch_pca_topk(const float *C, int n, int k, int iters, void *P, bool bf16_out, int64_t ld_p,
                           float *eigvals, void *ws, hipStream_t s) {
    const int p = pca_p(n, k), pp = pca_pp(n, k);
    const PcaLayout L = pca_layout(ws, n, k);
    const unsigned g = static_cast<unsigned>((static_cast<int64_t>(block_floats(n, pp)) + 255) / 256);
    hipLaunchKernelGGL(k_pca_init, dim3(g), dim3(256), 0, s, L.Q, n, p, pp);
    for (int it = 0; it < iters; ++it) {
        hipError_t e = launch_cq(L, C, n, pp, L.Q, L.Z, s);
        if (e != hipSuccess) return e;
        cholqr(L, n, p, pp, L.Z, L.Q, s);
    }
    // second orthonormalisation (CholQR2) into Z, then Rayleigh-Ritz on the
    // basis Z: Q = C Z, T = Z^T Q
    cholqr(L, n, p, pp, L.Q, L.Z, s);
    hipError_t e = launch_cq(L, C, n, pp, L.Z, L.Q, s);
    if (e != hipSuccess) return e;
    launch_gram(L.Z, L.Q, n, p, pp, L.part, s);
    const int chunks = sum_parts(L.part, gram_chunks(n), p, s);
    if (p <= 64)
        hipLaunchKernelGGL(k_jacobi_rot<64>, dim3(1), dim3(256), 0, s, L.part, chunks, p, L.rot, L.rounds, L.theta);
    else
        hipLaunchKernelGGL(k_jacobi_rot<kMaxP>, dim3(1), dim3(256), 0, s, L.part, chunks, p, L.rot, L.rounds,
                           L.theta);
    hipLaunchKernelGGL(k_jacobi_replay, dim3(static_cast<unsigned>(p)), dim3(kWave), 0, s, L.rot, L.rounds, p, L.Wt);
    // the Ritz vectors [k][n] overwrite Q (k <= pp)
    const dim3 ritz_grid(static_cast<unsigned>((n + 1023) / 1024), static_cast<unsigned>((k + kRitzE - 1) / kRitzE));
    hipLaunchKernelGGL(k_ritz, ritz_grid, dim3(256), 0, s, L.Z, n, p, pp, k, L.Wt, L.theta, L.Q, eigvals);
    if (bf16_out)
        hipLaunchKernelGGL(k_pca_out<bf16_bits>, dim3(static_cast<unsigned>(k)), dim3(256), 0, s, L.Q, n,
                           static_cast<bf16_bits *>(P), ld_p);
    else
        hipLaunchKernelGGL(k_pca_out<float>, dim3(static_cast<unsigned>(k)), dim3(256), 0, s, L.Q, n,
                           static_cast<float *>(P), ld_p);
    return hipGetLastError();
}

}  // namespace logra
