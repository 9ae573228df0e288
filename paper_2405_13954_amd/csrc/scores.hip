// Influence scores and per-query top-k (Sec. 2 Eq. (2) step (2); top-k most
// valuable training data, Sec. 4.1).
//
//   s[q][j] = sum_d te[q][d] * tr[j][d]      (fp32 accumulation)
//
// Score GEMM (bf16): one workgroup per 256 x 256 output tile; 4 waves, each
// owning a 128 x 128 quadrant as 4 x 4 blocks of 32x32x16 bf16 MFMAs (256
// fp32 accumulators per lane).  The contraction advances 64 at a time: the
// next slab of both operands is fetched with coalesced 128-bit loads into
// registers while the current slab is multiplied out of LDS, then stored
// into the other LDS buffer (one barrier per step).  LDS rows are padded to
// 144 bytes, which makes the lanes' 128-bit operand reads conflict-free.
// Tiles are ordered so that the workgroups sharing one 256-row train slab
// are dispatched together onto the same XCD (dispatch round-robins
// workgroups over the 8 XCDs), so the slab is fetched from HBM once into
// that XCD's L2.
//
// Top-k: one workgroup per query row.  An exact radix select (four 8-bit
// passes over order-preserving keys) finds the k-th largest score; one more
// pass collects the larger scores and the lowest-indexed ties in index order
// (block-wide prefix counts), and a bitonic sort orders them by (value desc,
// index asc).  With merge, the chunk's sorted list is merged with the
// caller's running list.
#include "common.h"
#include "internal.h"

namespace logra {
namespace {

#ifndef LOGRA_SC_SCHED
#define LOGRA_SC_SCHED 1   // interleave loads with the MFMA stream (scheduling hints)
#endif
#ifndef LOGRA_SC_NT
#define LOGRA_SC_NT 0      // non-temporal hint on the train-operand loads
#endif

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int LDR = BK + 8;       // padded LDS row (bf16 elements): 144 bytes
constexpr int GT = 256;           // GEMM threads
constexpr int kLoads = BM * BK / 8 / GT;   // 128-bit loads per operand and thread per slab
constexpr int kXcd = 8;

// One slab (BK columns) of both operands in flight, 128 bits per load.
struct Slab {
    u32x4 a[kLoads];
    u32x4 b[kLoads];
};

// scheduling-group masks of __builtin_amdgcn_sched_group_barrier
constexpr int kSchedMfma = 0x008, kSchedVmemRead = 0x020, kSchedDsRead = 0x100,
              kSchedDsWrite = 0x200;

__global__ __launch_bounds__(GT, 1) void k_scores_bf16(const bf16_bits *__restrict__ te, int64_t ld_te,
                                                       int Q, const bf16_bits *__restrict__ tr,
                                                       int64_t ld_tr, int64_t N, int D,
                                                       float *__restrict__ s, int64_t ld_s,
                                                       int m_tiles, int n_tiles) {
    __shared__ __attribute__((aligned(16))) bf16_bits As[2][BM * LDR];
    __shared__ __attribute__((aligned(16))) bf16_bits Bs[2][BN * LDR];

    // XCD-aware tile order: consecutive workgroups on one XCD share a train slab.
    const int bid = blockIdx.x;
    const int xcd = bid % kXcd, local = bid / kXcd;
    const int mt = local % m_tiles;
    const int nt = (local / m_tiles) * kXcd + xcd;
    if (nt >= n_tiles) return;
    const int m0 = mt * BM;
    const int64_t n0 = static_cast<int64_t>(nt) * BN;
    const int rows_a = Q - m0 < BM ? Q - m0 : BM;
    const int rows_b = N - n0 < BN ? static_cast<int>(N - n0) : BN;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // Buffer resources over this tile's rows (the host bounds rows * ld * 2 below
    // 2^31).  Load i of a thread covers row srow + 32 i, columns scol..scol+7 of
    // the slab; rows past the operand and columns past D read as zeros.
    const auto rsa = buf_rsrc_uniform(te + static_cast<int64_t>(m0) * ld_te,
                                      static_cast<uint32_t>(rows_a * ld_te * 2));
    const auto rsb = buf_rsrc_uniform(tr + n0 * ld_tr, static_cast<uint32_t>(rows_b * ld_tr * 2));
    const int srow = tid >> 3, scol = 8 * (tid & 7);
    uint32_t oa[kLoads], ob[kLoads];
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
        const int r = srow + 32 * i;
        oa[i] = r < rows_a ? static_cast<uint32_t>((r * ld_te + scol) * 2) : kBufOOB;
        ob[i] = r < rows_b ? static_cast<uint32_t>((r * ld_tr + scol) * 2) : kBufOOB;
    }
    auto gload = [&](Slab &st, int k0) {
        const bool kin = k0 + scol < D;
        const uint32_t dk = static_cast<uint32_t>(k0) * 2u;
#pragma unroll
        for (int i = 0; i < kLoads; ++i) {
            st.a[i] = buf_ld128(rsa, kin ? oa[i] + dk : kBufOOB);
#if LOGRA_SC_NT
            st.b[i] = buf_ld128_nt(rsb, kin ? ob[i] + dk : kBufOOB);
#else
            st.b[i] = buf_ld128(rsb, kin ? ob[i] + dk : kBufOOB);
#endif
        }
    };
    auto lstore = [&](const Slab &st, int buf) {
#pragma unroll
        for (int i = 0; i < kLoads; ++i) {
            *reinterpret_cast<u32x4 *>(&As[buf][(srow + 32 * i) * LDR + scol]) = st.a[i];
            *reinterpret_cast<u32x4 *>(&Bs[buf][(srow + 32 * i) * LDR + scol]) = st.b[i];
        }
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // Operand fragments: lane l reads row l % 32, contraction columns
    // 8 (l / 32) .. +8 of each 16-wide step.
    const int frow = lane & 31, fk = 8 * (lane >> 5);
    bf16x8 fa[2][4], fb[2][4];
    auto ldfrag = [&](int f, int buf, int ks) {
        const bf16_bits *Ab = &As[buf][(wm * 128 + frow) * LDR + fk + 16 * ks];
        const bf16_bits *Bb = &Bs[buf][(wn * 128 + frow) * LDR + fk + 16 * ks];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            fa[f][i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(Ab + i * 32 * LDR));
            fb[f][i] = as_bf16x8(*reinterpret_cast<const u32x4 *>(Bb + i * 32 * LDR));
        }
    };
    auto mfma_step = [&](int f) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = mfma32_bf16(fa[f][i], fb[f][j], acc[i][j]);
    };

    // One slab per half-step.  On entry LDS buffer `buf` holds slab kt and
    // `next` holds slab kt+1 in flight.  The half-step starts the loads of slab
    // kt+2 into `fill`, multiplies slab kt out of LDS (four 16-wide steps,
    // each step's fragments read while the previous step multiplies), stores
    // slab kt+1 into the other buffer and ends with the barrier.
    auto half = [&](int buf, Slab &fill, int kfill, const Slab &next) {
        gload(fill, kfill);
        ldfrag(0, buf, 0);
        ldfrag(1, buf, 1);
        mfma_step(0);
        ldfrag(0, buf, 2);
        mfma_step(1);
        ldfrag(1, buf, 3);
        mfma_step(0);
        lstore(next, buf ^ 1);
        mfma_step(1);
#if LOGRA_SC_SCHED
        // first fragments, then the 16 global loads over the first 32 MFMAs,
        // 8 fragment reads over each of the first three steps and the 16 LDS
        // stores over the last
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 8, 0);
#pragma unroll
        for (int ks = 0; ks < 3; ++ks) {
#pragma unroll
            for (int g = 0; g < 8; ++g) {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
                if (ks < 2) __builtin_amdgcn_sched_group_barrier(kSchedVmemRead, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, 8, 0);
        }
#pragma unroll
        for (int g = 0; g < 16; ++g) {
            __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
            __builtin_amdgcn_sched_group_barrier(kSchedDsWrite, 1, 0);
        }
#endif
        __syncthreads();
    };

    // The slab count is rounded up to even; slabs past D load as zeros.
    const int nk = (D + BK - 1) / BK;
    const int nk2 = nk + (nk & 1);
    Slab s0, s1;
    gload(s0, 0);
    gload(s1, BK);
    lstore(s0, 0);
    __syncthreads();
    for (int kt = 0; kt < nk2; kt += 2) {
        half(0, s0, (kt + 2) * BK, s1);
        half(1, s1, (kt + 3) * BK, s0);
    }

    // result register r of block (i, j): row 8*(r/4) + 4*(lane/32) + r%4, column lane%32
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row >= rows_a) continue;
            float *srow_p = s + static_cast<int64_t>(m0 + row) * ld_s + n0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int col = wn * 128 + j * 32 + (lane & 31);
                if (col < rows_b) srow_p[col] = acc[i][j][r];
            }
        }
}

// fp32 scores (small problems): one thread per score, sequential contraction.
__global__ __launch_bounds__(256) void k_scores_f32(const float *te, int64_t ld_te, int Q,
                                                    const float *tr, int64_t ld_tr, int64_t N, int D,
                                                    float *s, int64_t ld_s) {
    const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    const int q = blockIdx.y;
    if (j >= N) return;
    const float *a = te + static_cast<int64_t>(q) * ld_te;
    const float *b = tr + j * ld_tr;
    float acc = 0.f;
    for (int d = 0; d < D; ++d) acc = __builtin_fmaf(a[d], b[d], acc);
    s[static_cast<int64_t>(q) * ld_s + j] = acc;
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

// Exclusive block-wide prefix sum of v (0/1 flags); returns the prefix and
// writes the block total into *total.
__device__ __forceinline__ int block_scan(int v, int *warp_sums, int *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) warp_sums[wave] = x;
    __syncthreads();
    int base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < KT_THREADS / 64; ++w) {
        const int ws = warp_sums[w];
        if (w < wave) base += ws;
        tot += ws;
    }
    __syncthreads();
    *total = tot;
    return base + x - v;
}

__global__ __launch_bounds__(KT_THREADS) void k_topk(const float *__restrict__ S, int64_t ld_s,
                                                     int64_t N, int64_t base, int k,
                                                     float *__restrict__ val,
                                                     int64_t *__restrict__ idx, int merge) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t ck[kMaxTopk];
    __shared__ int64_t ci[kMaxTopk];
    __shared__ int warp_sums[KT_THREADS / 64];
    __shared__ uint32_t sh_prefix;
    __shared__ int sh_krem;

    const int q = blockIdx.x, tid = threadIdx.x;
    const float *row = S + static_cast<int64_t>(q) * ld_s;
    const int ksel = static_cast<int>(N < k ? N : k);   // candidates this chunk provides

    // 1. radix select of the ksel-th largest key
    uint32_t prefix = 0, pmask = 0;
    int krem = ksel;
    if (ksel > 0) {
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            hist[tid] = 0;
            __syncthreads();
            for (int64_t j = tid; j < N; j += KT_THREADS) {
                const uint32_t key = fkey(row[j]);
                if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
            }
            __syncthreads();
            if (tid == 0) {
                int cum = 0, d = 255;
                for (; d > 0; --d) {
                    if (cum + static_cast<int>(hist[d]) >= krem) break;
                    cum += static_cast<int>(hist[d]);
                }
                sh_prefix = prefix | (static_cast<uint32_t>(d) << shift);
                sh_krem = krem - cum;
            }
            __syncthreads();
            prefix = sh_prefix;
            krem = sh_krem;
            pmask |= 255u << shift;
            __syncthreads();
        }
    }
    // prefix is now the exact key of the ksel-th largest; krem ties of it are taken.
    const int ngt = ksel - krem;

    // 2. collect in index order: keys > prefix go to [0, ngt), the first krem
    //    keys == prefix go to [ngt, ksel).
    int seen_gt = 0, seen_eq = 0;
    if (ksel > 0) {
        for (int64_t j0 = 0; j0 < N; j0 += KT_THREADS) {
            const int64_t j = j0 + tid;
            uint32_t key = 0;
            if (j < N) key = fkey(row[j]);
            const int gt = (j < N && key > prefix) ? 1 : 0;
            const int eq = (j < N && key == prefix) ? 1 : 0;
            int tgt, teq;
            const int pg = block_scan(gt, warp_sums, &tgt);
            const int pe = block_scan(eq, warp_sums, &teq);
            if (gt) {
                ck[seen_gt + pg] = key;
                ci[seen_gt + pg] = base + j;
            }
            if (eq && seen_eq + pe < krem) {
                ck[ngt + seen_eq + pe] = key;
                ci[ngt + seen_eq + pe] = base + j;
            }
            seen_gt += tgt;
            seen_eq += teq;
            if (seen_gt >= ngt && seen_eq >= krem) break;   // uniform across the block
        }
    }
    // pad to a power of two >= k with (0, -1) entries (rank last)
    int P = 1;
    while (P < k) P <<= 1;
    for (int i = ksel + tid; i < P; i += KT_THREADS) {
        ck[i] = 0u;
        ci[i] = -1;
    }
    __syncthreads();

    // 3. bitonic sort by (key desc, index asc)
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < P; i += KT_THREADS) {
                const int jx = i ^ stride;
                if (jx > i) {
                    const bool up = (i & size) == 0;   // this run sorts "before"-first
                    const bool sw = up ? before(ck[jx], ci[jx], ck[i], ci[i])
                                       : before(ck[i], ci[i], ck[jx], ci[jx]);
                    if (sw) {
                        const uint32_t tk = ck[i];
                        ck[i] = ck[jx];
                        ck[jx] = tk;
                        const int64_t ti = ci[i];
                        ci[i] = ci[jx];
                        ci[jx] = ti;
                    }
                }
            }
            __syncthreads();
        }
    }

    // 4. write, merging with the caller's running list if asked
    float *vo = val + static_cast<int64_t>(q) * k;
    int64_t *io = idx + static_cast<int64_t>(q) * k;
    if (!merge) {
        for (int r = tid; r < k; r += KT_THREADS) {
            const bool ok = ci[r] >= 0;
            vo[r] = ok ? unkey(ck[r]) : -__builtin_huge_valf();
            io[r] = ok ? ci[r] : -1;
        }
        return;
    }
    // merged[r] from the two sorted lists (old: vo/io, new: ck/ci), staged in
    // LDS so that the old list is read completely before it is overwritten.
    __shared__ uint32_t mk[kMaxTopk];
    __shared__ int64_t mi[kMaxTopk];
    if (tid == 0) {
        int a = 0, b = 0;
        for (int r = 0; r < k; ++r) {
            const int64_t ia = a < k ? io[a] : -1;
            const uint32_t ka = ia >= 0 ? fkey(vo[a]) : 0u;
            const int64_t ib = b < k ? ci[b] : -1;
            const uint32_t kb = ib >= 0 ? ck[b] : 0u;
            if (before(ka, ia, kb, ib)) {
                mk[r] = ka;
                mi[r] = ia;
                ++a;
            } else {
                mk[r] = kb;
                mi[r] = ib;
                ++b;
            }
        }
    }
    __syncthreads();
    for (int r = tid; r < k; r += KT_THREADS) {
        const bool ok = mi[r] >= 0;
        vo[r] = ok ? unkey(mk[r]) : -__builtin_huge_valf();
        io[r] = ok ? mi[r] : -1;
    }
}

}  // namespace

hipError_t launch_scores(const void *te, int64_t ld_te, int Q, const void *tr, int64_t ld_tr,
                         int64_t N, int D, bool bf16, float *s, int64_t ld_s, hipStream_t st) {
    if (Q == 0 || N == 0) return hipSuccess;
    if (bf16) {
        const int m_tiles = (Q + BM - 1) / BM;
        const int n_tiles = static_cast<int>((N + BN - 1) / BN);
        const int n_groups = (n_tiles + kXcd - 1) / kXcd;
        const unsigned grid = static_cast<unsigned>(kXcd) * n_groups * m_tiles;
        hipLaunchKernelGGL(k_scores_bf16, dim3(grid), dim3(GT), 0, st,
                           static_cast<const bf16_bits *>(te), ld_te, Q,
                           static_cast<const bf16_bits *>(tr), ld_tr, N, D, s, ld_s, m_tiles, n_tiles);
    } else {
        const dim3 grid(static_cast<unsigned>((N + 255) / 256), static_cast<unsigned>(Q));
        hipLaunchKernelGGL(k_scores_f32, grid, dim3(256), 0, st, static_cast<const float *>(te), ld_te,
                           Q, static_cast<const float *>(tr), ld_tr, N, D, s, ld_s);
    }
    return hipGetLastError();
}

hipError_t launch_topk(const float *s, int64_t ld_s, int Q, int64_t N, int64_t base, int k,
                       float *val, int64_t *idx, bool merge, hipStream_t st) {
    if (Q == 0) return hipSuccess;
    hipLaunchKernelGGL(k_topk, dim3(Q), dim3(KT_THREADS), 0, st, s, ld_s, N, base, k, val, idx,
                       merge ? 1 : 0);
    return hipGetLastError();
}

}  // namespace logra
