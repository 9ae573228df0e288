// Self-influence of gradients, the normaliser of l-RelatIF (Sec. 4.2: each
// influence score is divided by the training example's own influence, which
// penalises outliers with large gradient norms):
//
//   self_j = sum_l g_jl^T (C_l + lambda_l I)^{-1} g_jl = sum_l |W_l g_jl|^2,
//   W_l = L_l^{-1},  C_l + lambda_l I = L_l L_l^T
//
// for a block-diagonal (per-layer) Hessian.  W_l comes from the damped
// Cholesky factor in float64 and is held as two bf16 arrays hi + lo (about
// 16 significant bits together), so the products run on the bf16 matrix
// cores with fp32 accumulation: y = g W_hi^T + g W_lo^T.
//
// bf16 gradients with D a multiple of 32: one workgroup per 256 gradients;
// for each block and each
// 256-wide pass over the output dimension, the contraction advances 32
// columns (one slab) per step: the slab of the gradients and of both W halves
// is fetched one step ahead into registers (range-checked buffer loads; rows
// and columns past the data read as zeros) and stored into one of two LDS
// buffers (80-byte rows, conflict-free fragment reads); 4 waves, each owning
// 128 gradients x 128 outputs as 4 x 4 blocks of 32x32x16 MFMAs.  After the
// last slab of a pass the squares of the outputs are summed over the wave's
// columns (registers, then DPP lane permutations inside rows of 16 lanes)
// into the gradients' running sums; at the end the partial sums are added
// through LDS, in a fixed order.
#include <type_traits>

#include "common.h"
#include "internal.h"


namespace logra {
namespace {

constexpr int SR = 256;                    // gradients per workgroup
constexpr int SO = 256;                    // output dimensions per pass
constexpr int SK = 32;                     // contraction columns per slab
constexpr int SLD = SK + 8;                // padded LDS row (bf16): 80 bytes
constexpr int STH = 256;                   // threads
constexpr int SL = SR * SK / 8 / STH;      // 128-bit loads per operand and thread per slab (4)

// DPP lane permutations within rows of 16 lanes (dpp_ctrl encodings)
constexpr int kDppXor1 = 0xB1;             // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;             // quad_perm [2, 3, 0, 1]
constexpr int kDppRowHalfMirror = 0x141;   // lane i <-> 7 - i within 8
constexpr int kDppRowMirror = 0x140;       // lane i <-> 15 - i within 16

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}

typedef f32x16 Acc[4][4];   // one wave's 128 x 128 result quadrant (4 x 4 blocks of 32 x 32)

__device__ __forceinline__ void zero_acc(Acc &acc) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
}

// After the last slab of an output pass: the squared outputs, summed over
// the lane's four column blocks, then reduce-scattered over the 16 lanes of
// each DPP row in four halvings (partners l ^ 15, l ^ 7, l ^ 2, l ^ 1, all
// within the row; each lane keeps the half selected by the bit in which it
// differs from its partner), so that each lane ends with 4 of the 64 row
// entries e = 16 i + r (block i, register r) summed over the row's 16
// columns: psum[s] += entry 4 (lane % 16) + s.  Lanes l and l ^ 16 hold the
// two halves of the same rows' sums.  Clears the accumulators.
__device__ __forceinline__ void fold_rows(Acc &acc, float (&psum)[4], int lane) {
    const bool b3 = lane & 8, b2 = lane & 4, b1 = lane & 2, b0 = lane & 1;
    auto sq = [&](int e) {
        const int i = e >> 4, r = e & 15;
        float v = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) v = __builtin_fmaf(acc[i][j][r], acc[i][j][r], v);
        return v;
    };
    float u[32], w[16], x[8];
#pragma unroll
    for (int k = 0; k < 32; ++k) {
        const float lo = sq(k), hi = sq(32 + k);
        u[k] = (b3 ? hi : lo) + dpp_f<kDppRowMirror>(b3 ? lo : hi);
        __builtin_amdgcn_sched_barrier(0);   // a few accumulators in VGPRs at a time
    }
#pragma unroll
    for (int k = 0; k < 16; ++k)
        w[k] = (b2 ? u[16 + k] : u[k]) + dpp_f<kDppRowHalfMirror>(b2 ? u[k] : u[16 + k]);
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = (b1 ? w[8 + k] : w[k]) + dpp_f<kDppXor2>(b1 ? w[k] : w[8 + k]);
#pragma unroll
    for (int k = 0; k < 4; ++k) psum[k] += (b0 ? x[4 + k] : x[k]) + dpp_f<kDppXor1>(b0 ? x[k] : x[4 + k]);
    zero_acc(acc);
}

// Adds the partial row sums of the workgroup's 256 gradients -- two column
// halves (waves wn = 0, 1) x the two 16-lane rows of each half-wave --
// through LDS (rowsum: 4 x 256 floats) in a fixed order and writes the
// results.  Ends with the workgroup's last barrier.
__device__ __forceinline__ void finish_rows(const float (&psum)[4], float *rowsum, int tid, int lane, int wm,
                                            int wn, int nrows, int64_t r0, float *self_out, float *rsqrt_out) {
    const int h16 = (lane >> 4) & 1;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int e = 4 * (lane & 15) + k, i = e >> 4, r = e & 15;
        rowsum[(2 * wn + h16) * 256 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)] = psum[k];
    }
    __syncthreads();
    if (tid < nrows) {
        const float sv = (rowsum[tid] + rowsum[256 + tid]) + (rowsum[512 + tid] + rowsum[768 + tid]);
        if (self_out) self_out[r0 + tid] = sv;
        if (rsqrt_out) rsqrt_out[r0 + tid] = sv > 0.f ? 1.0f / sqrtf(sv) : 0.f;
    }
}

struct Slab3 {
    u32x4 a[SL], h[SL], l[SL];
};

__global__ __launch_bounds__(STH, 1) void k_self_influence(const bf16_bits *__restrict__ g, int64_t ld,
                                                           int64_t rows, int D, int n_blocks,
                                                           const bf16_bits *__restrict__ w_hi,
                                                           const bf16_bits *__restrict__ w_lo,
                                                           float *__restrict__ self_out,
                                                           float *__restrict__ rsqrt_out) {
    __shared__ __attribute__((aligned(16))) bf16_bits As[2][SR * SLD];
    __shared__ __attribute__((aligned(16))) bf16_bits Hs[2][SO * SLD];
    __shared__ __attribute__((aligned(16))) bf16_bits Ls[2][SO * SLD];
    __shared__ float rowsum[2][2][SR];

    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * SR;
    const int nrows = rows - r0 < SR ? static_cast<int>(rows - r0) : SR;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int n_ot = (D + SO - 1) / SO;
    const int Dp = n_ot * SO;        // rows of each W half, zero past D
    const int ns = (D + SK - 1) / SK;
    const int ns2 = ns + (ns & 1);   // slabs per output pass, rounded up to even (extra slabs load zeros)

    // staging: load i of a thread covers row (or output) srow + 64 i, columns scol..scol+7
    const int srow = tid >> 2, scol = 8 * (tid & 3);
    const auto rsa = buf_rsrc_uniform(g + r0 * ld, static_cast<uint32_t>(nrows * ld * 2));
    uint32_t oa[SL];
#pragma unroll
    for (int i = 0; i < SL; ++i) {
        const int r = srow + 64 * i;
        oa[i] = r < nrows ? static_cast<uint32_t>((r * ld + scol) * 2) : kBufOOB;
    }
    // load cursor: slab (ls, lot, ll) = (contraction slab, output pass, block),
    // advanced by one slab per gload in the order the slabs are consumed
    int ls = 0, lot = 0, ll = 0;
    auto gload = [&](Slab3 &st) {
        const bool live = ll < n_blocks && ls < ns;   // uniform (D is a multiple of SK)
        const int col = ls * SK + scol;
        const bool cin = live;
        const uint32_t da = static_cast<uint32_t>((static_cast<int64_t>(ll) * D + ls * SK) * 2);
        const size_t wblk = static_cast<size_t>(live ? ll : 0) * Dp * D;
        const auto rh = buf_rsrc_uniform(w_hi + wblk, static_cast<uint32_t>(Dp * D * 2));
        const auto rl = buf_rsrc_uniform(w_lo + wblk, static_cast<uint32_t>(Dp * D * 2));
#pragma unroll
        for (int i = 0; i < SL; ++i) {
            const int o = lot * SO + srow + 64 * i;   // output dimension = row of W (zero rows past D)
            const uint32_t ow = cin ? static_cast<uint32_t>((o * D + col) * 2) : kBufOOB;
            st.a[i] = buf_ld128(rsa, cin ? oa[i] + da : kBufOOB);
            st.h[i] = buf_ld128(rh, ow);
            st.l[i] = buf_ld128(rl, ow);
        }
        if (++ls == ns2) {
            ls = 0;
            if (++lot == n_ot) {
                lot = 0;
                ++ll;
            }
        }
    };
    auto lstore = [&](const Slab3 &st, int buf) {
#pragma unroll
        for (int i = 0; i < SL; ++i) {
            const int off = (srow + 64 * i) * SLD + scol;
            *reinterpret_cast<u32x4 *>(&As[buf][off]) = st.a[i];
            *reinterpret_cast<u32x4 *>(&Hs[buf][off]) = st.h[i];
            *reinterpret_cast<u32x4 *>(&Ls[buf][off]) = st.l[i];
        }
    };

    Acc acc;
    float psum[4] = {0.f, 0.f, 0.f, 0.f};   // row sums (fold_rows)
    zero_acc(acc);

    // fragments: lane l reads row (l % 32) of each 32-row block, columns
    // 8 (l / 32) .. +8 of each 16-wide step
    const int frow = lane & 31, fk = 8 * (lane >> 5);
    auto compute = [&](int buf) {
#pragma unroll
        for (int ks = 0; ks < SK / 16; ++ks) {
            bf16x8 fa[4], fh[4], fl[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                fa[i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(
                    &As[buf][(wm * 128 + i * 32 + frow) * SLD + fk + 16 * ks]));
                fh[i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(
                    &Hs[buf][(wn * 128 + i * 32 + frow) * SLD + fk + 16 * ks]));
                fl[i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(
                    &Ls[buf][(wn * 128 + i * 32 + frow) * SLD + fk + 16 * ks]));
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc[i][j] = mfma32_bf16(fa[i], fh[j], acc[i][j]);
                    acc[i][j] = mfma32_bf16(fa[i], fl[j], acc[i][j]);
                }
            __builtin_amdgcn_sched_barrier(0);   // one step's fragments live at a time
        }
    };
    // One slab in flight in registers while the previous one is multiplied out
    // of LDS (the prefetch runs across pass and block boundaries, in the order
    // of the cursor).
    Slab3 st;
    gload(st);
    lstore(st, 0);
    __syncthreads();
    for (int l = 0; l < n_blocks; ++l)
        for (int ot = 0; ot < n_ot; ++ot) {
            for (int k = 0; k < ns2; k += 2) {
                gload(st);
                compute(0);
                lstore(st, 1);
                __syncthreads();
                gload(st);
                compute(1);
                lstore(st, 0);
                __syncthreads();
            }
            fold_rows(acc, psum, lane);
        }

    finish_rows(psum, &rowsum[0][0][0], tid, lane, wm, wn, nrows, r0, self_out, rsqrt_out);
}

// ------------------------------------------------------------------------
// bf16 gradients with D a multiple of 64: the same 256 x 256 tile per pass,
// 4 waves x (4 x 4 32x32x16 MFMA blocks), with the operands copied straight
// from memory into an LDS ring (gfx950 buffer_load ... lds), as in the score
// GEMM.  The contraction of a pass runs over 2D columns of the interleaved W
// (per 64-column chunk c: hi, then lo), one 64-column step at a time; the
// gradients' 64 columns of chunk c serve both steps of the chunk, so a
// gradient slab is copied once per two steps.  Ring: 2 gradient stages, 3 W
// stages of 32 KB (256 rows of 128 bytes, chunk c of row r at position
// c ^ ((r >> 1) & 7)).  Copies run two steps ahead: during the first step of
// a chunk, the next chunk's gradient slab and the W slab two steps ahead;
// during the second, the W slab two steps ahead.  One barrier per step, in
// the middle of its last 16-wide MFMA group, after each wave has waited for
// its own copies of the next step's slabs (vmcnt, which counts the copies).
constexpr int DBK = 64;                          // columns per step
constexpr int kDSlab = 256 * DBK * 2;            // bytes of one operand slab
constexpr int kDStA = 2, kDStB = 3;
constexpr int kDLdsB = kDStA * kDSlab;
constexpr int kDLds = (kDStA + kDStB) * kDSlab;  // 160 KB
constexpr int kDCopies = kDSlab / 1024 / 4;      // 1 KB copies per wave and operand slab (8)

__global__ __launch_bounds__(STH, 1) void k_self_influence_dma(const bf16_bits *__restrict__ g, int64_t ld,
                                                               int64_t rows, int D, int n_blocks,
                                                               const bf16_bits *__restrict__ w,
                                                               float *__restrict__ self_out,
                                                               float *__restrict__ rsqrt_out) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[kDLds];

    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * SR;
    const int nrows = rows - r0 < SR ? static_cast<int>(rows - r0) : SR;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const uint32_t lds0 = lds_addr(smem);
    const int n_ot = (D + SO - 1) / SO;
    const int Dp = n_ot * SO;
    const int n_chunks = D / DBK;            // gradient slabs per pass (two W steps each)
    const int n_steps = 2 * n_chunks;        // W steps per pass
    const uint32_t w_row = 2u * D * 2u;      // bytes per row of the interleaved W

    // copy i of this wave covers rows rb + 8 i, rb = 64 wave + (l >> 3), of a
    // slab; lane l loads chunk (l & 7) ^ (((8 wave + i) * 4 + (l >> 4)) & 7) of
    // its row.  Byte offsets are va[i & 1] + i * (8 rows), plus the slab's
    // column offset: two per-lane bases per operand.  Rows at or past nrows
    // lie past the gradient buffer's range and read zeros; so does every copy
    // past the last block, through a descriptor of size 0.
    const int rb = 64 * wave + (lane >> 3);
    uint32_t va[2], vb[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int cc = 8 * ((lane & 7) ^ ((4 * h + (lane >> 4)) & 7));
        va[h] = static_cast<uint32_t>((rb * ld + cc) * 2);
        vb[h] = static_cast<uint32_t>(rb) * w_row + static_cast<uint32_t>(cc) * 2u;
    }
    const uint32_t a_bytes = static_cast<uint32_t>(nrows * ld * 2);
    const uint32_t a_step8 = static_cast<uint32_t>(8 * ld * 2), b_step8 = 8u * w_row;
    // issue cursors, advanced in the order the slabs are consumed: gradient
    // slab (al, aot, aj) and W step (bl, bot, bt) = (block, output pass, chunk
    // or step within the pass)
    int al = 0, aot = 0, aj = 0, bl = 0, bot = 0, bt = 0;
    auto rsrc_a = [&]() { return buf_rsrc_uniform(g + r0 * ld, al < n_blocks ? a_bytes : 0u); };
    auto issue_a = [&](const __amdgpu_buffer_rsrc_t &rsa, uint32_t lds, int i) {
        const uint32_t dk = static_cast<uint32_t>((al * D + aj * DBK) * 2) + i * a_step8;
        // the streamed gradients carry the non-temporal hint (1% faster on a 200,000-row
        // store; the same hint on the inverse-factor copies was slower)
        copy_to_lds_nt(rsa, va[i & 1] + dk, lds + wave * kDCopies * 1024 + i * 1024);
    };
    auto next_a = [&]() {
        if (++aj == n_chunks) {
            aj = 0;
            if (++aot == n_ot) {
                aot = 0;
                ++al;
            }
        }
    };
    auto rsrc_b = [&]() {
        const size_t blk = static_cast<size_t>(bl < n_blocks ? bl : 0) * Dp * 2 * D;
        return buf_rsrc_uniform(w + blk, bl < n_blocks ? static_cast<uint32_t>(Dp) * w_row : 0u);
    };
    auto issue_b = [&](const __amdgpu_buffer_rsrc_t &rsb, uint32_t lds, int i) {
        const uint32_t dk = static_cast<uint32_t>(bot * SO) * w_row + static_cast<uint32_t>(bt * DBK * 2) + i * b_step8;
        copy_to_lds(rsb, vb[i & 1] + dk, lds + wave * kDCopies * 1024 + i * 1024);
    };
    auto next_b = [&]() {
        if (++bt == n_steps) {
            bt = 0;
            if (++bot == n_ot) {
                bot = 0;
                ++bl;
            }
        }
    };

    // fragment byte offsets inside a slab: lane l reads row (l % 32) of each
    // 32-row block, logical chunk 2 ks + (l / 32) at position chunk ^ sw
    const int sw = (lane >> 1) & 7;
    const uint32_t fa0 = (wm * 128 + (lane & 31)) * 128, fb0 = (wn * 128 + (lane & 31)) * 128;
    uint32_t fo[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) fo[ks] = static_cast<uint32_t>(((2 * ks + (lane >> 5)) ^ sw) * 16);

    Acc acc;
    float psum[4] = {0.f, 0.f, 0.f, 0.f};
    zero_acc(acc);
    bf16x8 fa[2][4], fb[2][4];
    // fragment read q (0..7) of a 16-wide step: A block q/2 for even q, B block q/2 for odd q
    auto ldfrag1 = [&](int f, const uint8_t *abase, const uint8_t *bbase, int ks, int q) {
        const int i = q >> 1;
        if (q & 1)
            fb[f][i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(bbase + fb0 + fo[ks] + i * 4096));
        else
            fa[f][i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(abase + fa0 + fo[ks] + i * 4096));
    };
    auto mfma1 = [&](int f, int idx) {
        const int i = idx >> 2, j = idx & 3;
        acc[i][j] = mfma32_bf16(fa[f][i], fb[f][j], acc[i][j]);
    };

    // One step: W slab t (stage sb) against the gradient slab of its chunk
    // (stage sa).  FIRST (first step of a chunk): also copies the next
    // gradient slab, into the other A stage, whose previous slab was last
    // read in the step before this one.
    int sa = 0, sb = 0;
    auto step = [&](auto first_tag) {
        constexpr bool FIRST = decltype(first_tag)::value;
        const uint8_t *abase = smem + sa * kDSlab, *bbase = smem + kDLdsB + sb * kDSlab;
        const int nb1 = sb == 2 ? 0 : sb + 1;   // stage of W step t + 1
        const int nb2 = sb == 0 ? 2 : sb - 1;   // stage of W step t + 2 (held step t - 1)
        const int na = FIRST ? sa : sa ^ 1;     // gradient stage of step t + 1
        const uint32_t la = lds0 + (sa ^ 1) * kDSlab, lb = lds0 + kDLdsB + nb2 * kDSlab;
        const auto rsa = rsrc_a();
        const auto rsb = rsrc_b();
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ks = 0; ks < 3; ++ks) {
            const int f = ks & 1;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                mfma1(f, 2 * q);
                mfma1(f, 2 * q + 1);
                if (ks == 0 && FIRST) issue_a(rsa, la, q);
                if (ks == 1) issue_b(rsb, lb, q);
                ldfrag1(f ^ 1, abase, bbase, ks + 1, q);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if (FIRST) next_a();
        next_b();
#pragma unroll
        for (int m = 0; m < 8; ++m) mfma1(1, m);
        __builtin_amdgcn_sched_barrier(0);
        // outstanding copies allowed: this step's (A + B after a FIRST step, B after a second)
        if (FIRST)
            asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(2 * kDCopies) : "memory");
        else
            asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(kDCopies) : "memory");
        const uint8_t *nabase = smem + na * kDSlab, *nbbase = smem + kDLdsB + nb1 * kDSlab;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            ldfrag1(0, nabase, nbbase, 0, q);
            mfma1(1, 8 + q);
            __builtin_amdgcn_sched_barrier(0);
        }
        sa = na;
        sb = nb1;
    };

    {   // prologue: gradient slab 0, W steps 0 and 1
        const auto rsa0 = rsrc_a();
        const auto rsb0 = rsrc_b();
#pragma unroll
        for (int q = 0; q < 8; ++q) issue_a(rsa0, lds0, q);
        next_a();
#pragma unroll
        for (int q = 0; q < 8; ++q) issue_b(rsb0, lds0 + kDLdsB, q);
        next_b();
        const auto rsb1 = rsrc_b();
#pragma unroll
        for (int q = 0; q < 8; ++q) issue_b(rsb1, lds0 + kDLdsB + kDSlab, q);
        next_b();
    }
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" :: "n"(kDCopies) : "memory");
#pragma unroll
    for (int q = 0; q < 8; ++q) ldfrag1(0, smem, smem + kDLdsB, 0, q);
    for (int l = 0; l < n_blocks; ++l)
        for (int ot = 0; ot < n_ot; ++ot) {
            for (int c = 0; c < n_chunks; ++c) {
                step(std::integral_constant<bool, true>());
                step(std::integral_constant<bool, false>());
            }
            fold_rows(acc, psum, lane);
        }
    // the copies past the last block are still in flight
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    finish_rows(psum, reinterpret_cast<float *>(smem), tid, lane, wm, wn, nrows, r0, self_out, rsqrt_out);
}

// Any D (and fp32 gradients): one workgroup per gradient; thread d forms
// output d of W_l g_l with the hi + lo halves (all D columns), a fixed-order
// block sum adds the squares, blocks in order.  For small problems.
template <typename TIn>
__global__ __launch_bounds__(256) void k_self_influence_rows(const TIn *__restrict__ g, int64_t ld, int D,
                                                             int n_blocks, const bf16_bits *__restrict__ w_hi,
                                                             const bf16_bits *__restrict__ w_lo,
                                                             float *__restrict__ self_out,
                                                             float *__restrict__ rsqrt_out) {
    __shared__ float red[256];
    const int64_t j = blockIdx.x;
    const int tid = threadIdx.x;
    const int Dp = (D + 255) / 256 * 256;
    float total = 0.f;
    for (int l = 0; l < n_blocks; ++l) {
        const TIn *gl = g + j * ld + static_cast<int64_t>(l) * D;
        float part = 0.f;
        for (int d = tid; d < D; d += 256) {
            const bf16_bits *h = w_hi + (static_cast<size_t>(l) * Dp + d) * D;
            const bf16_bits *lo = w_lo + (static_cast<size_t>(l) * Dp + d) * D;
            float y = 0.f;
            for (int k = 0; k < D; ++k)
                y = __builtin_fmaf(bf16_to_f32(h[k]) + bf16_to_f32(lo[k]), static_cast<float>(load_in_d<TIn>(gl + k)), y);
            part = __builtin_fmaf(y, y, part);
        }
        red[tid] = part;
        __syncthreads();
        for (int w = 128; w > 0; w >>= 1) {
            if (tid < w) red[tid] += red[tid + w];
            __syncthreads();
        }
        if (tid == 0) total += red[0];
        __syncthreads();
    }
    if (tid == 0) {
        if (self_out) self_out[j] = total;
        if (rsqrt_out) rsqrt_out[j] = total > 0.f ? 1.0f / sqrtf(total) : 0.f;
    }
}

}  // namespace

hipError_t launch_self_influence(const void *g, bool bf16, int64_t ld, int64_t rows, int D, int n_blocks,
                                 const void *ws, float *self_out, float *rsqrt_out, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    void *w = const_cast<void *>(ws);
    const bf16_bits *hi = self_influence_w(w, D, n_blocks, false), *lo = self_influence_w(w, D, n_blocks, true);
    if (self_influence_interleaved(bf16, D)) {
        const unsigned grid = static_cast<unsigned>((rows + SR - 1) / SR);
        hipLaunchKernelGGL(k_self_influence_dma, dim3(grid), dim3(STH), 0, s, static_cast<const bf16_bits *>(g),
                           ld, rows, D, n_blocks, hi, self_out, rsqrt_out);
    } else if (bf16 && D % SK == 0) {
        const unsigned grid = static_cast<unsigned>((rows + SR - 1) / SR);
        hipLaunchKernelGGL(k_self_influence, dim3(grid), dim3(STH), 0, s, static_cast<const bf16_bits *>(g), ld,
                           rows, D, n_blocks, hi, lo, self_out, rsqrt_out);
    } else if (bf16) {
        hipLaunchKernelGGL(k_self_influence_rows<bf16_bits>, dim3(static_cast<unsigned>(rows)), dim3(256), 0, s,
                           static_cast<const bf16_bits *>(g), ld, D, n_blocks, hi, lo, self_out, rsqrt_out);
    } else {
        hipLaunchKernelGGL(k_self_influence_rows<float>, dim3(static_cast<unsigned>(rows)), dim3(256), 0, s,
                           static_cast<const float *>(g), ld, D, n_blocks, hi, lo, self_out, rsqrt_out);
    }
    return hipGetLastError();
}

}  // namespace logra
