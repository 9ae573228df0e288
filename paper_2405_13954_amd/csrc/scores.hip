// Influence scores and per-query top-k (Sec. 2 Eq. (2) step (2); top-k most
// valuable training data, Sec. 4.1).
//
//   s[q][j] = sum_d te[q][d] * tr[j][d]      (fp32 result)
//
// Score GEMM (bf16, fp32 accumulation): one workgroup per 256 x 256 output tile; 4 waves, each
// owning a 128 x 128 quadrant as 4 x 4 blocks of 32x32x16 bf16 MFMAs (256
// fp32 accumulators per lane), 64 contraction columns (one slab) per step.
// Tiles are ordered so that the workgroups sharing one 256-row train slab are
// dispatched together onto the same XCD (dispatch round-robins workgroups
// over the 8 XCDs), so the slab is fetched from HBM once into that XCD's L2.
// Operands are copied straight from memory into an LDS ring with gfx950's
// buffer_load ... lds (no register staging); the issue order of MFMAs,
// copies and fragment reads is fixed by hand.  fp32 / fp64 operands take a
// float64-accumulating tiled kernel.
//
// Top-k: one workgroup per query row.  An exact radix select (four 8-bit
// passes over order-preserving keys) finds the k-th largest score; when more
// scores tie at it than are needed, a second radix select over the
// (complemented) indices keeps the lowest-indexed ones.  The selected
// entries are sorted by (value desc, index asc) with a bitonic sort and, with
// merge, merged with the caller's running list.  For long chunks the GEMM
// epilogue filters: only scores at or above a per-query threshold (the k-th
// value of a running list that already covers a prefix of the chunk, hence
// a lower bound on the final k-th value) are appended to candidate lists, and
// the selection runs over those; a list that overflows falls back to the
// query's full score row.
#include "common.h"
#include "internal.h"

namespace logra {
namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int GT = 256;           // GEMM threads
constexpr int kXcd = 8;

// Epilogue of a 256 x 256 tile: the fp32 scores, times the optional row and
// column scales (s * row_scale[q] * col_scale[j], for normalised scores), go
// to s (rows past Q and columns past N are skipped).  With a filter, scores at
// or above the row's threshold are also appended to the row's top-k candidate
// list; the count keeps growing past the capacity so that an overflow is
// visible.  Each half-wave of one (i, r) step holds one row, so candidates
// are counted with ballots: a first pass writes the scores and each (row,
// column half)'s count to LDS, one global atomic per row reserves the tile's
// space, and a second pass places each candidate at its reserved base plus its
// ballot prefix (in column order within a column half).  `lds` is 5 KB of free
// LDS (thresholds, counts and bases).
__device__ __forceinline__ void store_scores(const f32x16 (&acc)[4][4], float *lds, float *__restrict__ s,
                                             int64_t ld_s, int m0, int64_t n0, int rows_a, int rows_b,
                                             int wm, int wn, int tid, int lane, const ScoreFilter &filt,
                                             const ScoreScale &scale) {
    const bool filter = filt.thr != nullptr;
    float *ths = lds;                                        // [256] row thresholds
    int *cnt = reinterpret_cast<int *>(lds + 256);           // [2][256] candidates per column half
    int *base = reinterpret_cast<int *>(lds + 768);          // [2][256] first slot per column half
    if (filter) {
        ths[tid] = tid < rows_a ? filt.thr[m0 + tid] : __builtin_inff();
        __syncthreads();
    }
    const uint64_t half = lane < 32 ? 0xffffffffull : 0xffffffff00000000ull;   // the lanes of this row
    auto value = [&](int i, int r, int j, float rs, int col) {   // the same in both passes
        float v = acc[i][j][r];
        if (scale.row) v *= rs;
        if (scale.col && col < rows_b) v *= scale.col[n0 + col];
        return v;
    };
    // result register r of block (i, j): row 8*(r/4) + 4*(lane/32) + r%4, column lane%32
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row >= rows_a) continue;
            const int64_t q = m0 + row;
            float *srow_p = s + q * ld_s + n0;
            const float t = filter ? ths[row] : 0.f;
            const float rs = scale.row ? scale.row[q] : 1.f;
            int hits = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = wn * 128 + j * 32 + (lane & 31);
                const float v = value(i, r, j, rs, col);
                if (col < rows_b) srow_p[col] = v;
                if (filter) hits += __popcll(__builtin_amdgcn_ballot_w64(col < rows_b && v >= t) & half);
            }
            if (filter && (lane & 31) == 0) cnt[wn * 256 + row] = hits;
        }
    if (!filter) return;
    __syncthreads();
    if (tid < rows_a) {
        const int c0 = cnt[tid], c1 = cnt[256 + tid];
        const int b = c0 + c1 > 0 ? atomicAdd(filt.cnt + m0 + tid, c0 + c1) : 0;
        base[tid] = b;
        base[256 + tid] = b + c0;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row >= rows_a) continue;
            const int64_t q = m0 + row;
            const float t = ths[row];
            const float rs = scale.row ? scale.row[q] : 1.f;
            int pos = base[wn * 256 + row];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = wn * 128 + j * 32 + (lane & 31);
                const float v = value(i, r, j, rs, col);
                const bool hit = col < rows_b && v >= t;
                const uint64_t m = __builtin_amdgcn_ballot_w64(hit) & half;
                if (hit) {
                    const int p = pos + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                            static_cast<uint32_t>(m >> 32),
                                            __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u)));
                    if (p < filt.cap) {
                        filt.val[q * filt.cap + p] = v;
                        filt.idx[q * filt.cap + p] = static_cast<int>(n0) + col;
                    }
                }
                pos += __popcll(m);
            }
        }
}

// ------------------------------------------------------------------------
// Score GEMM with asynchronous global->LDS copies (gfx950 buffer_load ... lds).
// The operands travel from memory straight into LDS (no register staging, no
// LDS store instructions).  The LDS ring holds three slabs of the train operand, which
// streams from HBM and is copied two slabs ahead, and two slabs of the test
// operand, which the L2 mostly serves and is copied one slab ahead
// (3 x 32 KB + 2 x 32 KB = 160 KB).  The train copies carry the
// non-temporal hint: the streamed rows are evicted first, so the test operand
// (re-read by every train tile) stays in the caches longer.  One barrier per slab: each wave waits
// for its own copies of the slab, the barrier makes every wave's copies
// visible and frees the stages of the previous slab, and the next copies are
// issued before the slab is multiplied.
//
// LDS layout of an operand slab: 256 rows of 128 bytes (8 chunks of 16 B);
// chunk c of row r is stored at position c ^ ((r >> 1) & 7), which makes the
// 16 lanes of each quarter-wave fragment read (16 consecutive rows, one chunk)
// hit 16 different 16-byte bank groups.  A copy instruction writes a
// contiguous 1 KB (8 whole rows, so every request is a full 128-byte line):
// lane l stores row (l >> 3), position (l & 7).
constexpr int kSlabOp = BM * BK * 2;         // bytes of one operand slab (32 KB)
constexpr int kStagesA = 2, kStagesB = 3;
constexpr int kLdsB = kStagesA * kSlabOp;    // B stages follow the A stages
constexpr int kLdsBytes = (kStagesA + kStagesB) * kSlabOp;
constexpr int kCopies = kSlabOp / 1024 / 4;  // 1 KB copies per wave and operand per slab (8)

__global__ __launch_bounds__(GT, 1) void k_scores_dma(const bf16_bits *__restrict__ te, int64_t ld_te,
                                                      int Q, const bf16_bits *__restrict__ tr,
                                                      int64_t ld_tr, int64_t N, int D,
                                                      float *__restrict__ s, int64_t ld_s,
                                                      int m_tiles, int n_tiles, ScoreFilter filt,
                                                       ScoreScale scale) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[kLdsBytes];

    const int bid = blockIdx.x;
    const int xcd = bid % kXcd, local = bid / kXcd;
    const int mt = local % m_tiles;
    const int nt = (local / m_tiles) * kXcd + xcd;
    if (nt >= n_tiles) return;
    const int m0 = mt * BM;
    const int64_t n0 = static_cast<int64_t>(nt) * BN;
    const int rows_a = Q - m0 < BM ? Q - m0 : BM;
    const int rows_b = N - n0 < BN ? static_cast<int>(N - n0) : BN;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    // LDS byte address of the ring (the address-space cast yields the 32-bit LDS offset)
    const uint32_t lds0 = static_cast<uint32_t>(
        reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t *)smem));

    const auto rsa = buf_rsrc_uniform(te + static_cast<int64_t>(m0) * ld_te,
                                      static_cast<uint32_t>(rows_a * ld_te * 2));
    const auto rsb = buf_rsrc_uniform(tr + n0 * ld_tr, static_cast<uint32_t>(rows_b * ld_tr * 2));
    // copy i of this wave covers rows (8 wave + i) * 8 .. +8 of an operand slab;
    // lane l loads chunk (l & 7) ^ (((8 wave + i) * 4 + (l >> 4)) & 7) of its row
    uint32_t oa[kCopies], ob[kCopies];
    int ccol[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) ccol[h] = 8 * ((lane & 7) ^ ((4 * h + (lane >> 4)) & 7));
#pragma unroll
    for (int i = 0; i < kCopies; ++i) {
        const int r = (wave * kCopies + i) * 8 + (lane >> 3);
        oa[i] = r < rows_a ? static_cast<uint32_t>((r * ld_te + ccol[i & 1]) * 2) : kBufOOB;
        ob[i] = r < rows_b ? static_cast<uint32_t>((r * ld_tr + ccol[i & 1]) * 2) : kBufOOB;
    }
    auto issue = [&](const __amdgpu_buffer_rsrc_t &rs, const uint32_t(&o)[kCopies], int slab, uint32_t lds) {
        const int k0 = slab * BK;
        const uint32_t dk = static_cast<uint32_t>(k0) * 2u;
        const bool kin0 = k0 + ccol[0] < D, kin1 = k0 + ccol[1] < D;
        const uint32_t la = lds + wave * kCopies * 1024;
#pragma unroll
        for (int i = 0; i < kCopies; ++i)
            copy_to_lds(rs, ((i & 1) ? kin1 : kin0) ? o[i] + dk : kBufOOB, la + i * 1024);
    };

    // fragment byte offsets inside an operand slab: lane l reads row (l % 32) of
    // each 32-row block, logical chunk 2 ks + (l / 32) at position chunk ^ sw
    const int sw = (lane >> 1) & 7;
    const uint32_t fa0 = (wm * 128 + (lane & 31)) * 128, fb0 = (wn * 128 + (lane & 31)) * 128;
    uint32_t fo[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) fo[ks] = static_cast<uint32_t>(((2 * ks + (lane >> 5)) ^ sw) * 16);

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    bf16x8 fa[2][4], fb[2][4];
    // fragment read g (0..7) of a 16-wide step: A block g/2 for even g, B block g/2 for odd g
    auto ldfrag1 = [&](int f, const uint8_t *abase, const uint8_t *bbase, int ks, int g) {
        const int i = g >> 1;
        if (g & 1)
            fb[f][i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(bbase + fb0 + fo[ks] + i * 4096));
        else
            fa[f][i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(abase + fa0 + fo[ks] + i * 4096));
    };
    auto mfma1 = [&](int f, int idx) {
        const int i = idx >> 2, j = idx & 3;
        acc[i][j] = mfma32_bf16(fa[f][i], fb[f][j], acc[i][j]);
    };

    // Slab kt lives in A stage kt % 2 and B stage kt % 3.  Before slab kt
    // is read, the copies in flight are (A kt, B kt+1), issued during slab
    // kt-1, and B kt from before; waiting until at most kCopies remain leaves
    // only B kt+1 (issued last).  The wait and the barrier sit in the middle
    // of the previous slab's last 16-wide step: its first 8 MFMAs cover the
    // barrier, its last 8 cover the reads of the new slab's first fragments.
    // (lgkmcnt(0) first: this wave's reads of the stages that the next copies
    // overwrite are complete before any wave passes the barrier.)  The step
    // is issued in a fixed order (scheduling barriers): groups of two MFMAs
    // with one copy of the next slabs and one fragment read of the next
    // 16-wide step.
    const int nk = (D + BK - 1) / BK;
    issue(rsa, oa, 0, lds0);
    issue(rsb, ob, 0, lds0 + kLdsB);
    issue(rsb, ob, 1, lds0 + kLdsB + kSlabOp);
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" :: "n"(kCopies) : "memory");
#pragma unroll
    for (int g = 0; g < 8; ++g) ldfrag1(0, smem, smem + kLdsB, 0, g);
    int sa = 0, sb = 0;   // stages of slab kt
    for (int kt = 0; kt < nk; ++kt) {
        const int na = sa ^ 1, nb2 = sb == 0 ? 2 : sb - 1;   // stages of A kt+1 and B kt+2
        const int nb1 = sb == 2 ? 0 : sb + 1;                // stage of B kt+1
        const uint8_t *abase = smem + sa * kSlabOp, *bbase = smem + kLdsB + sb * kSlabOp;
        const uint32_t dka = static_cast<uint32_t>((kt + 1) * BK) * 2u, dkb = dka + BK * 2u;
        const bool ka0 = (kt + 1) * BK + ccol[0] < D, ka1 = (kt + 1) * BK + ccol[1] < D;
        const bool kb0 = (kt + 2) * BK + ccol[0] < D, kb1 = (kt + 2) * BK + ccol[1] < D;
        const uint32_t la = lds0 + na * kSlabOp + wave * kCopies * 1024;
        const uint32_t lb = lds0 + kLdsB + nb2 * kSlabOp + wave * kCopies * 1024;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ks = 0; ks < 3; ++ks) {
            const int f = ks & 1;
#pragma unroll
            for (int g = 0; g < 8; ++g) {
                mfma1(f, 2 * g);
                mfma1(f, 2 * g + 1);
                if (ks == 0)
                    copy_to_lds(rsa, ((g & 1) ? ka1 : ka0) ? oa[g] + dka : kBufOOB, la + g * 1024);
                else if (ks == 1)
                    copy_to_lds_nt(rsb, ((g & 1) ? kb1 : kb0) ? ob[g] + dkb : kBufOOB, lb + g * 1024);
                ldfrag1(f ^ 1, abase, bbase, ks + 1, g);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int m = 0; m < 8; ++m) mfma1(1, m);
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(kCopies) : "memory");
        const uint8_t *nabase = smem + na * kSlabOp, *nbbase = smem + kLdsB + nb1 * kSlabOp;
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            ldfrag1(0, nabase, nbbase, 0, g);
            mfma1(1, 8 + g);
            __builtin_amdgcn_sched_barrier(0);
        }
        sa = na;
        sb = nb1;
    }
    // the copies of the slabs past the end are still in flight
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    store_scores(acc, reinterpret_cast<float *>(smem), s, ld_s, m0, n0, rows_a, rows_b, wm, wn, tid,
                 lane, filt, scale);
}

// fp32 / fp64 operands: every product and sum in float64 (a product of two
// fp32 values is exact there), the result rounded once to fp32.  One 64 x 64
// output tile per workgroup; 16-column slabs of both operands are staged
// through LDS as float64 (coalesced row reads, transposed stores), and each
// thread accumulates a 4 x 4 block over the whole contraction in order d =
// 0, 1, ..., D-1.  Scales (normalised scores) multiply in float64 before the
// rounding.
constexpr int FT = 64, FK = 16;
template <typename TA, typename TB>
__global__ __launch_bounds__(256) void k_scores_f64acc(const TA *te, int64_t ld_te, int Q, const TB *tr,
                                                       int64_t ld_tr, int64_t N, int D, float *s, int64_t ld_s,
                                                       ScoreScale scale) {
    __shared__ double As[FK][FT + 1];   // [column][query]
    __shared__ double Bs[FK][FT + 1];   // [column][train row]
    const int q0 = blockIdx.y * FT;
    const int64_t j0 = static_cast<int64_t>(blockIdx.x) * FT;
    const int tid = threadIdx.x, ta = tid >> 4, tb = tid & 15;
    double acc[4][4] = {};
    for (int k0 = 0; k0 < D; k0 += FK) {
#pragma unroll
        for (int u = 0; u < FT * FK / 256; ++u) {
            const int e = tid + 256 * u, r = e / FK, c = e % FK, d = k0 + c;
            const int q = q0 + r;
            const int64_t j = j0 + r;
            As[c][r] = (q < Q && d < D) ? load_in_d<TA>(te + static_cast<int64_t>(q) * ld_te + d) : 0.0;
            Bs[c][r] = (j < N && d < D) ? load_in_d<TB>(tr + j * ld_tr + d) : 0.0;
        }
        __syncthreads();
#pragma unroll
        for (int c = 0; c < FK; ++c) {
            double x[4], y[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                x[u] = As[c][4 * ta + u];
                y[u] = Bs[c][tb + 16 * u];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[u][v] = fma(x[u], y[v], acc[u][v]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int q = q0 + 4 * ta + u;
        if (q >= Q) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int64_t j = j0 + tb + 16 * v;   // consecutive threads: consecutive columns
            if (j >= N) continue;
            double val = acc[u][v];
            if (scale.row) val *= static_cast<double>(scale.row[q]);
            if (scale.col) val *= static_cast<double>(scale.col[j]);
            s[static_cast<int64_t>(q) * ld_s + j] = static_cast<float>(val);
        }
    }
}

// ---------------------------------------------------------------- top-k --
constexpr int KT_THREADS = 256;

// Order-preserving map float -> uint32 (larger float <=> larger key); -0.0
// maps to the key of +0.0 so that equal values tie.
__device__ __forceinline__ uint32_t fkey(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float unkey(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// (key a, idx a) ranks before (key b, idx b); idx < 0 is padding, ranks last.
__device__ __forceinline__ bool before(uint32_t ka, int64_t ia, uint32_t kb, int64_t ib) {
    if (ia < 0) return false;
    if (ib < 0) return true;
    if (ka != kb) return ka > kb;
    return ia < ib;
}

// Sources of a selection: a row of scores (local index = column), or a
// row's candidate list (local index = the candidate's column).  Global index
// = base + local index.
struct RowSrc {
    const float *row;
    int64_t n;
    int64_t base;
    __device__ int64_t size() const { return n; }
    __device__ float value(int64_t j) const { return row[j]; }
    __device__ uint32_t local(int64_t j) const { return static_cast<uint32_t>(j); }
    __device__ int64_t global(int64_t j) const { return base + j; }
};
struct CandSrc {
    const float *v;
    const int *c;
    int64_t n;
    int64_t base;
    __device__ int64_t size() const { return n; }
    __device__ float value(int64_t j) const { return v[j]; }
    __device__ uint32_t local(int64_t j) const { return static_cast<uint32_t>(c[j]); }
    __device__ int64_t global(int64_t j) const { return base + c[j]; }
};

struct TopkShared {
    uint32_t hist[256];
    uint32_t ck[kMaxTopk];
    int64_t ci[kMaxTopk];
    uint32_t mk[kMaxTopk];
    int64_t mi[kMaxTopk];
    uint32_t prefix;
    int rem;
    uint32_t neq;
    int count;
};

// Radix select (four 8-bit digits, most significant first) of the `want`-th
// largest key(j) over the j < n with in(j).  Returns that key; *rem = how many
// elements equal to it belong to the `want` largest, *neq = how many exist.
template <class KeyFn, class InFn>
__device__ uint32_t radix_select(int64_t n, KeyFn key, InFn in, int want, TopkShared &sh, int *rem,
                                 uint32_t *neq) {
    const int tid = threadIdx.x;
    uint32_t prefix = 0, pmask = 0;
    int r = want;
    uint32_t eq = 0;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        sh.hist[tid] = 0;
        __syncthreads();
        for (int64_t j = tid; j < n; j += KT_THREADS) {
            if (!in(j)) continue;
            const uint32_t kk = key(j);
            if ((kk & pmask) == prefix) atomicAdd(&sh.hist[(kk >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (tid == 0) {
            int cum = 0, d = 255;
            for (; d > 0; --d) {
                if (cum + static_cast<int>(sh.hist[d]) >= r) break;
                cum += static_cast<int>(sh.hist[d]);
            }
            sh.prefix = prefix | (static_cast<uint32_t>(d) << shift);
            sh.rem = r - cum;
            sh.neq = sh.hist[d];
        }
        __syncthreads();
        prefix = sh.prefix;
        r = sh.rem;
        eq = sh.neq;
        pmask |= 255u << shift;
        __syncthreads();
    }
    *rem = r;
    *neq = eq;
    return prefix;
}

// Top-k of one source, merged with the running list (vo, io) when `merge`.
// The k-th largest key is found by radix select; when more elements tie at
// it than are needed, a second radix select over the complemented local
// index keeps the lowest-indexed ones.  Exactly min(n, k) elements are then
// collected (in any order), padded to a power of two and sorted by (value
// descending, index ascending).
template <class Src>
__device__ void topk_row(const Src &src, int k, float *vo, int64_t *io, bool merge, TopkShared &sh) {
    const int tid = threadIdx.x;
    const int64_t n = src.size();
    const int ksel = static_cast<int>(n < k ? n : k);
    uint32_t kth = 0, idx_limit = 0xffffffffu;
    if (ksel > 0) {
        int rem;
        uint32_t neq;
        kth = radix_select(
            n, [&](int64_t j) { return fkey(src.value(j)); }, [](int64_t) { return true; }, ksel, sh,
            &rem, &neq);
        if (neq > static_cast<uint32_t>(rem)) {
            int rem2;
            uint32_t neq2;
            const uint32_t c = radix_select(
                n, [&](int64_t j) { return ~src.local(j); },
                [&](int64_t j) { return fkey(src.value(j)) == kth; }, rem, sh, &rem2, &neq2);
            idx_limit = ~c;
        }
    }
    if (tid == 0) sh.count = 0;
    __syncthreads();
    if (ksel > 0) {
        for (int64_t j = tid; j < n; j += KT_THREADS) {
            const uint32_t kk = fkey(src.value(j));
            if (kk > kth || (kk == kth && src.local(j) <= idx_limit)) {
                const int pos = atomicAdd(&sh.count, 1);
                sh.ck[pos] = kk;
                sh.ci[pos] = src.global(j);
            }
        }
    }
    // pad to a power of two >= k with (0, -1) entries (rank last)
    int P = 1;
    while (P < k) P <<= 1;
    __syncthreads();
    for (int i = ksel + tid; i < P; i += KT_THREADS) {
        sh.ck[i] = 0u;
        sh.ci[i] = -1;
    }
    __syncthreads();

    // bitonic sort by (key desc, index asc)
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < P; i += KT_THREADS) {
                const int jx = i ^ stride;
                if (jx > i) {
                    const bool up = (i & size) == 0;   // this run sorts "before"-first
                    const bool sw = up ? before(sh.ck[jx], sh.ci[jx], sh.ck[i], sh.ci[i])
                                       : before(sh.ck[i], sh.ci[i], sh.ck[jx], sh.ci[jx]);
                    if (sw) {
                        const uint32_t tk = sh.ck[i];
                        sh.ck[i] = sh.ck[jx];
                        sh.ck[jx] = tk;
                        const int64_t ti = sh.ci[i];
                        sh.ci[i] = sh.ci[jx];
                        sh.ci[jx] = ti;
                    }
                }
            }
            __syncthreads();
        }
    }

    if (!merge) {
        for (int r = tid; r < k; r += KT_THREADS) {
            const bool ok = sh.ci[r] >= 0;
            vo[r] = ok ? unkey(sh.ck[r]) : -__builtin_huge_valf();
            io[r] = ok ? sh.ci[r] : -1;
        }
        return;
    }
    // merged[r] from the two sorted lists (old: vo/io, new: ck/ci), staged in
    // LDS so that the old list is read completely before it is overwritten.
    if (tid == 0) {
        int a = 0, b = 0;
        for (int r = 0; r < k; ++r) {
            const int64_t ia = a < k ? io[a] : -1;
            const uint32_t ka = ia >= 0 ? fkey(vo[a]) : 0u;
            const int64_t ib = b < k ? sh.ci[b] : -1;
            const uint32_t kb = ib >= 0 ? sh.ck[b] : 0u;
            if (before(ka, ia, kb, ib)) {
                sh.mk[r] = ka;
                sh.mi[r] = ia;
                ++a;
            } else {
                sh.mk[r] = kb;
                sh.mi[r] = ib;
                ++b;
            }
        }
    }
    __syncthreads();
    for (int r = tid; r < k; r += KT_THREADS) {
        const bool ok = sh.mi[r] >= 0;
        vo[r] = ok ? unkey(sh.mk[r]) : -__builtin_huge_valf();
        io[r] = ok ? sh.mi[r] : -1;
    }
}

// One workgroup per query row over a full row of scores.
__global__ __launch_bounds__(KT_THREADS) void k_topk(const float *__restrict__ S, int64_t ld_s,
                                                     int64_t N, int64_t base, int k,
                                                     float *__restrict__ val,
                                                     int64_t *__restrict__ idx, int merge) {
    __shared__ TopkShared sh;
    const int q = blockIdx.x;
    const RowSrc src{S + static_cast<int64_t>(q) * ld_s, N, base};
    topk_row(src, k, val + static_cast<int64_t>(q) * k, idx + static_cast<int64_t>(q) * k, merge != 0,
             sh);
}

// Threshold of each row for candidate filtering: the k-th value of the
// running list (-inf while it holds fewer than k entries); clears the row's
// candidate count.
__global__ __launch_bounds__(256) void k_topk_threshold(const float *__restrict__ val,
                                                        const int64_t *__restrict__ idx, int Q, int k,
                                                        float *__restrict__ thr, int *__restrict__ cnt) {
    const int q = blockIdx.x * 256 + threadIdx.x;
    if (q >= Q) return;
    const int64_t last = static_cast<int64_t>(q) * k + k - 1;
    thr[q] = idx[last] >= 0 ? val[last] : -__builtin_huge_valf();
    cnt[q] = 0;
}

// Merge of each row's candidates into its running list; a row whose
// candidates overflowed the capacity is selected from its full score row.
__global__ __launch_bounds__(KT_THREADS) void k_topk_filtered(
    const float *__restrict__ S, int64_t ld_s, int64_t N, int64_t base, int k, float *__restrict__ val,
    int64_t *__restrict__ idx, const int *__restrict__ cnt, const float *__restrict__ cval,
    const int *__restrict__ cidx, int cap) {
    __shared__ TopkShared sh;
    const int q = blockIdx.x;
    float *vo = val + static_cast<int64_t>(q) * k;
    int64_t *io = idx + static_cast<int64_t>(q) * k;
    const int c = cnt[q];
    if (c <= cap) {
        const CandSrc src{cval + static_cast<int64_t>(q) * cap, cidx + static_cast<int64_t>(q) * cap, c,
                          base};
        topk_row(src, k, vo, io, true, sh);
    } else {
        const RowSrc src{S + static_cast<int64_t>(q) * ld_s, N, base};
        topk_row(src, k, vo, io, true, sh);
    }
}

}  // namespace

hipError_t launch_scores(const void *te, int te_dt, int64_t ld_te, int Q, const void *tr, int tr_dt,
                         int64_t ld_tr, int64_t N, int D, float *s, int64_t ld_s, const ScoreFilter *filt,
                         const ScoreScale &scale, hipStream_t st) {
    if (Q == 0 || N == 0) return hipSuccess;
    if (te_dt == kBF16 && tr_dt == kBF16) {
        const int m_tiles = (Q + BM - 1) / BM;
        const int n_tiles = static_cast<int>((N + BN - 1) / BN);
        const int n_groups = (n_tiles + kXcd - 1) / kXcd;
        const unsigned grid = static_cast<unsigned>(kXcd) * n_groups * m_tiles;
        const ScoreFilter none{nullptr, nullptr, nullptr, nullptr, 0};
        hipLaunchKernelGGL(k_scores_dma, dim3(grid), dim3(GT), 0, st, static_cast<const bf16_bits *>(te), ld_te, Q,
                           static_cast<const bf16_bits *>(tr), ld_tr, N, D, s, ld_s, m_tiles, n_tiles,
                           filt ? *filt : none, scale);
        return hipGetLastError();
    }
    if (filt || te_dt == kBF16 || tr_dt == kBF16) return hipErrorInvalidValue;   // bf16 pairs only with bf16
    const dim3 grid(static_cast<unsigned>((N + FT - 1) / FT), static_cast<unsigned>((Q + FT - 1) / FT));
    auto go = [&](auto a, auto b) {
        using TA = decltype(a);
        using TB = decltype(b);
        hipLaunchKernelGGL((k_scores_f64acc<TA, TB>), grid, dim3(256), 0, st, static_cast<const TA *>(te), ld_te, Q,
                           static_cast<const TB *>(tr), ld_tr, N, D, s, ld_s, scale);
        return hipGetLastError();
    };
    if (te_dt == kF64) return tr_dt == kF64 ? go(double{}, double{}) : go(double{}, float{});
    return tr_dt == kF64 ? go(float{}, double{}) : go(float{}, float{});
}

int64_t topk_prefix_rows(int64_t N, int k) {
    // Expected candidates past a prefix of P rows: about k (N - P) / P; aim
    // for at most half the capacity.
    int64_t P = (2 * static_cast<int64_t>(k) * N + kCandCap - 1) / kCandCap;
    if (P < 4096) P = 4096;
    P = (P + 255) / 256 * 256;
    return 2 * P <= N ? P : 0;
}

hipError_t launch_topk(const float *s, int64_t ld_s, int Q, int64_t N, int64_t base, int k,
                       float *val, int64_t *idx, bool merge, hipStream_t st) {
    if (Q == 0) return hipSuccess;
    hipLaunchKernelGGL(k_topk, dim3(Q), dim3(KT_THREADS), 0, st, s, ld_s, N, base, k, val, idx,
                       merge ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_topk_threshold(const float *val, const int64_t *idx, int Q, int k, float *thr,
                                 int *cnt, hipStream_t st) {
    if (Q == 0) return hipSuccess;
    hipLaunchKernelGGL(k_topk_threshold, dim3((Q + 255) / 256), dim3(256), 0, st, val, idx, Q, k, thr,
                       cnt);
    return hipGetLastError();
}

hipError_t launch_topk_filtered(const float *s, int64_t ld_s, int Q, int64_t N, int64_t base, int k,
                                float *val, int64_t *idx, const int *cnt, const float *cval,
                                const int *cidx, int cap, hipStream_t st) {
    if (Q == 0) return hipSuccess;
    hipLaunchKernelGGL(k_topk_filtered, dim3(Q), dim3(KT_THREADS), 0, st, s, ld_s, N, base, k, val, idx,
                       cnt, cval, cidx, cap);
    return hipGetLastError();
}

}  // namespace logra
