// Fused per-example structured gradient projection (LoGra, Sec. 3.1, Eq. (5)).
//
//   G_b = sum_t m_bt (P_out dy_bt)(P_in x_bt)^T        (k_out x k_in, fp32)
//
// The work of a layer group is cut into uniform items, so that every
// workgroup streams about the same number of bytes whatever the layer widths
// and the padding (layers differ up to 4x in bytes per token; half of the
// tiles of a ragged batch are empty):
//
//  0. k_project_prep: clears the work counter and, for masked inputs, builds
//     the ordered list of 64-token tiles holding at least one valid token,
//     each with the 64-bit set of its valid tokens (and every tile's set, by
//     tile index, for step B).
//  A. k_project_chunks (persistent, sized to the resident capacity): one item
//     = one contraction chunk (<= 6144 columns at k <= 32, <= 14336 above) of one side (x or dy) of one
//     listed tile.  Layers given the same x tensor (q/k/v, gate/up of a
//     transformer block) share their x items: one pass over the chunk feeds
//     up to three projections P_in (k <= 32), each with the same per-element
//     sums as a pass of its own.  Workgroups take items from an atomic counter as they
//     finish (items differ up to 4x in columns and workgroups in speed, so a
//     static assignment leaves a long tail).  Each of the four waves streams
//     a contiguous band of the chunk's columns (whole bands read HBM faster
//     than steps dealt round-robin); each lane feeds a 128-bit buffer load straight into its
//     MFMA operand (row = token for x/dy, row = projection dimension for P;
//     16x16x32 bf16 or 16x16x4 fp32, fp32 accumulation).  Masked tokens, rows
//     of P beyond k and lanes past the chunk end get an out-of-range offset:
//     they read zeros without a memory access or a branch, so NaN/Inf in
//     padding cannot leak.  The waves' partial x'/dy' are folded in a fixed
//     order and written, in the MFMA result layout, to the workspace.  A
//     workgroup claims its next item when it starts one, so the claim's
//     round trip is hidden behind the stream.
//  B. k_project_tile_finish: per tile, x' and dy' are the fixed-order sums of
//     their chunk partials; the tile's sum over tokens of dy'_t x'_t^T is then
//     formed by fp32 MFMAs straight from those sums (one wave per 16 x 16 block
//     of G at k <= 16; at k > 16 one workgroup per tile, x' and dy' read once
//     into LDS).  Empty tiles give 0.
//  C. k_project_reduce: per example and 16 x 16 block of G, the tile sums are
//     added in tile order and G_b is written (fp32 or bf16, round to nearest
//     even) to the caller's store row.
// Every sum has a fixed order, so results are bitwise reproducible.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace logra {
namespace {

constexpr int MB = 4;                     // 16-token row blocks per tile
constexpr int TT = 16 * MB;               // tokens per tile
static_assert(TT == 64, "a tile's valid-token set is one 64-bit word");
constexpr int NW = 4;                     // waves per workgroup
constexpr int kMaxSlots = 256;            // chunk slots a group can order by width
static_assert(kMaxSlots <= 1024 && kMaxGroup <= 64, "an ordered slot packs its slot into 10 bits, its layer into 6");
constexpr int NT = NW * kWave;            // threads per workgroup

// Contraction columns per work item: 14,336, one item per layer side of a
// Llama3-8B block.  At k > 32 it measured best of 2,048..14,336.  At k <= 16
// 6,144 was best while every item wrote chunk partials; with one chunk per
// side the stream kernel pairs a tile's two sides and writes no partials, and
// 14,336 took the 28-layer Llama3-8B launch from 782 to 721 us (the
// shared-input one from 722 to 675 us).
constexpr int kChunkCols = 14336;
__host__ __device__ constexpr int chunk_cols(int) { return kChunkCols; }
// Register pipeline depth of the register-staged path.
__host__ __device__ constexpr int stages_for(int KT) { return KT >= 4 ? 2 : 3; }

constexpr int kMaxShare = 3;   // layers projected from one pass over a shared x

// Rounds of items (one item per workgroup) at the end of a launch that a
// workgroup claims only when it is free; before them it claims its next item
// when it starts one.
constexpr int kAheadRounds = 2;
// The streamed x / dy copies of the per-wave DMA path carry the non-temporal
// hint up to this KT (k <= 32): it leaves the cache to the projection
// matrices.  Measured: the 7-layer k = 16 launch 7% faster.
constexpr int kDmaNtMaxKT = 2;
constexpr int kDmaCols = 64;     // columns per step: 128 bytes of a bf16 row
constexpr int kLdsBytes = 160 * 1024;
template <int KT, int S>
struct DmaShape {
    static constexpr int kX = TT / 8;                // copies of the x slab (8 token rows of 128 B each)
    static constexpr int kPm = 2 * KT;               // copies of one P slab (8 rows each)
    static constexpr int kCopies = kX + S * kPm;
    static constexpr int kStage = kCopies * 1024;    // bytes of one stage
    static constexpr int kFold = MB * S * KT * kWave * 16;   // one wave's results (f32x4 per lane)
    // ring stages per wave: three when the workgroup's LDS allows, else two
    static constexpr int kStages = NW * 3 * kStage <= kLdsBytes ? 3 : 2;
    static constexpr int kWaveRing = kStages * kStage;       // bytes per wave
    static constexpr int kRing = NW * kWaveRing;             // bytes per workgroup
    // a wave's fold fits its ring, and 1 KB is left for the workgroup's other LDS
    static constexpr bool kFits = kRing + 1024 <= kLdsBytes && kFold <= kWaveRing;
};
template <int KT, int S, typename TIn>
__host__ __device__ constexpr bool use_dma() {
    return sizeof(TIn) == 2 && DmaShape<KT, S>::kFits;
}

struct ChunkLayer {     // 56 bytes: 48 of them fit the kernel arguments
    const void *x;
    const void *dy;
    const void *p_in;
    const void *p_out;
    int n_in, n_out;
    uint32_t part_unit;   // first float of this layer's chunk partials, in units of 1024 floats
    uint16_t c_in, c_out;  // chunks of the x side and of the dy side (partial slots per tile)
    uint16_t x_items;      // x-side work slots: c_in for the first layer of a shared x, else 0
    uint16_t slot_begin;   // work slots of the layers before this one
    uint8_t share_n;       // layers whose x' this layer's x items produce (itself first)
    uint8_t share[kMaxShare];
};
static_assert(sizeof(ChunkLayer) == 56, "the layer table stays within the kernel arguments");
constexpr int kPartUnit = 1024;   // floats per tile per chunk at KT = 1 (every layer's partials are a multiple)
__device__ __forceinline__ float *part_of(float *part, const ChunkLayer &L) {
    return part + static_cast<size_t>(L.part_unit) * kPartUnit;
}

struct ProjArgs {
    ChunkLayer layer[kMaxGroup];
    int n_layers;
    int slots;      // chunk slots of all layers
    int ordered;    // slot_order holds the processing order of the slots
    int paired;
    // paired (every layer side one chunk): item 2 p + s is side s (0 = x, 1 = dy)
    // of pair p = (layer, listed tile) in the stream kernel, of unit p = (layer,
    // group of four listed tiles) in the tile-group kernel; slot_order holds each
    // layer's x slot, widest pair first; the tile sums are formed in the kernel
    // processing order: entry = layer << 10 | work slot (over all layers)
    alignas(4) uint16_t slot_order[kMaxSlots];
    const uint8_t *mask;
    const int *tiles;     // non-empty tiles (b * tpe + tile) in index order; NULL = all
    const uint64_t *bits; // their valid tokens (bit i = token 64 tile + i), beside tiles
    const uint64_t *tile_bits;   // the valid tokens of every tile b * tpe + tile (masked inputs)
    const int *n_tiles;   // their count (device), read when tiles != NULL
    int *work;            // items handed out beyond the first gridDim.x (device counter)
    float *part;    // chunk partials, MFMA result layout, TT x 16KT floats each
    float *gpart;   // per-tile sums [layer][b][tile][16 KT x 16 KT], 16 x 16 blocks in the MFMA result layout
    int B, T, tpe;  // tpe = tiles per example
    int k_in, k_out, ck;
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
__device__ __forceinline__ void mma_step(f32x4 (&acc)[MB][KT], const u32x4 (&xa)[MB],
                                         const u32x4 (&pb)[KT], bf16_bits) {
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int j = 0; j < KT; ++j) acc[m][j] = mfma16_bf16(as_bf16x8(xa[m]), as_bf16x8(pb[j]), acc[m][j]);
}

template <int KT>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[MB][KT], const u32x4 (&xa)[MB],
                                         const u32x4 (&pb)[KT], float) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int j = 0; j < KT; ++j)
                acc[m][j] = mfma16_f32(__uint_as_float(xa[m][e]), __uint_as_float(pb[j][e]), acc[m][j]);
}

// One wave's share of  A'_s[TT x 16KT] = A[TT x nk] * P_s[k x nk]^T for the
// S projections P_s (s < S) of one operand A (a shared input: one pass over
// A; a missing P_s reads zeros), A and P_s with row strides lda and ldp.
// Each wave takes a contiguous band of the contraction steps (bf16: of
// 64-column units, two steps each, see step_of).  Every load is unconditional
// (out-of-range offsets read zeros), and the ST-stage register pipeline
// keeps ST-1 steps in flight while a step multiplies.  Each wave's step
// count is rounded up to a multiple of ST with empty steps (no memory access,
// zero operands), so the loop body has no exits.  Result column block
// s * KT + j of acc holds block j of A'_s.
template <int KT, int S, typename TIn, int ST>
__device__ __forceinline__ void project_part(f32x4 (&acc)[MB][S * KT], const TIn *A, int lda,
                                             const TIn *const (&P)[S], int ldp, int nk, int k,
                                             const bool (&tok_ok)[MB], int wave, int lane) {
    constexpr int E = InTraits<TIn>::kElems;
    constexpr int SS = InTraits<TIn>::kStep;
    constexpr uint32_t ES = sizeof(TIn);
    const int row = lane & 15;
    const int kg = lane >> 4;
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int j = 0; j < S * KT; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int nsteps = (nk + SS - 1) / SS;
    // the wave's j-th step, in its band of units: for bf16 a unit is two
    // 32-column steps (a 64-column step of project_part_dma, so that both
    // paths add the same products in the same order); for fp32 one step.
    // Steps past the wave's count (the rounding of the pipeline) read zeros.
    constexpr bool kPairs = sizeof(TIn) == 2;
    constexpr int kNone = 1 << 24;   // a step index past any chunk
    const int units = kPairs ? (nsteps + 1) / 2 : nsteps;
    const int per = (units + NW - 1) / NW;
    const int first = wave * per;
    const int count = max(0, min(per, units - first)) * (kPairs ? 2 : 1);
    auto step_of = [&](int j) {
        return j >= count ? kNone : kPairs ? 2 * (first + (j >> 1)) + (j & 1) : first + j;
    };
    if (count == 0) return;

    const auto ra = buf_rsrc(A, (static_cast<uint32_t>(TT - 1) * lda + nk) * ES);
    __amdgpu_buffer_rsrc_t rp[S];
#pragma unroll
    for (int q = 0; q < S; ++q)
        rp[q] = buf_rsrc(P[q] ? P[q] : A, P[q] ? (static_cast<uint32_t>(k - 1) * ldp + nk) * ES : 0u);
    uint32_t aoff[MB], poff[KT];
#pragma unroll
    for (int m = 0; m < MB; ++m)
        aoff[m] = tok_ok[m] ? (static_cast<uint32_t>(16 * m + row) * lda + kg * E) * ES : kBufOOB;
#pragma unroll
    for (int j = 0; j < KT; ++j)
        poff[j] = (16 * j + row < k) ? (static_cast<uint32_t>(16 * j + row) * ldp + kg * E) * ES : kBufOOB;

    auto load = [&](int st, u32x4(&xa)[MB], u32x4(&pb)[S * KT]) {
        const bool in_k = st * SS + kg * E < nk;   // false past the last step: all lanes zero
        const uint32_t koff = static_cast<uint32_t>(st * SS) * ES;
#pragma unroll
        for (int m = 0; m < MB; ++m)
            xa[m] = buf_ld128(ra, in_k ? aoff[m] + koff : kBufOOB);
#pragma unroll
        for (int q = 0; q < S; ++q)
#pragma unroll
            for (int j = 0; j < KT; ++j) pb[q * KT + j] = buf_ld128(rp[q], in_k ? poff[j] + koff : kBufOOB);
    };

    const int iters = (count + ST - 1) / ST;
    u32x4 xa[ST][MB], pb[ST][S * KT];
#pragma unroll
    for (int i = 0; i < ST - 1; ++i) load(step_of(i), xa[i], pb[i]);
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < ST; ++i) {
            load(step_of(it * ST + i + ST - 1), xa[(i + ST - 1) % ST], pb[(i + ST - 1) % ST]);
            mma_step<S * KT>(acc, xa[i], pb[i], TIn{});
        }
    }
}

// project_part for bf16 operands, staged through the wave's own
// LDS ring instead of registers.  A step is 64 columns: the x slab (64 tokens
// x 128 bytes) and one P slab (16 KT rows x 128 bytes) per projection, each
// copy instruction moving 8 whole rows (full 128-byte lines) from memory
// straight into LDS (gfx950 buffer_load ... lds).  Row r of a slab sits at
// byte 128 r with its 16-byte chunk c at position c ^ (r & 7); the copies
// give lane l rows 8 q + l / 8 (so r & 7 = l / 8) and position l & 7, which
// makes the lane's source chunk (l & 7) ^ (l / 8) the same in every copy.  A
// fragment read (ds_read_b128) hands lane (row, kg) the 8 elements of chunk
// 4 h + kg of its row for half-step h.  The ring keeps all but one of its
// stages in flight (three stages where the LDS allows, else two); the wave waits only on its own copies (s_waitcnt vmcnt) and
// shares nothing with the other waves, so no barrier is needed.  Masked
// tokens, rows of P beyond k and columns past the chunk read zeros (an
// out-of-range offset).  The wave's steps are a contiguous band of the
// chunk; prefetches past the band are all out of range and keep the copy
// count of every iteration the same.
template <int KT, int S>
__device__ __forceinline__ void project_part_dma(f32x4 (&acc)[MB][S * KT], const bf16_bits *A, int lda,
                                                 const bf16_bits *const (&P)[S], int ldp, int nk, int k,
                                                 uint64_t valid, int wave, int lane, const uint8_t *ring,
                                                 uint32_t ring_addr) {
    using Sh = DmaShape<KT, S>;
    constexpr int NS = Sh::kStages;
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int j = 0; j < S * KT; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int nsteps = (nk + kDmaCols - 1) / kDmaCols;
    const int per = (nsteps + NW - 1) / NW;   // each wave streams a contiguous band of steps
    const int first = wave * per;
    const int mine = max(0, min(per, nsteps - first));
    if (mine == 0) return;
    const auto ra = buf_rsrc(A, (static_cast<uint32_t>(TT - 1) * lda + nk) * 2u);
    __amdgpu_buffer_rsrc_t rp[S];
#pragma unroll
    for (int q = 0; q < S; ++q)   // a missing projection reads zeros
        rp[q] = buf_rsrc(P[q] ? P[q] : A, P[q] ? (static_cast<uint32_t>(k - 1) * ldp + nk) * 2u : 0u);
    const int sub = lane >> 3;
    const int lcol = ((lane & 7) ^ sub) * 8;         // the lane's element column within a step
    uint32_t xo[Sh::kX], po[Sh::kPm];
#pragma unroll
    for (int q = 0; q < Sh::kX; ++q) {
        const int t = 8 * q + sub;
        xo[q] = (valid >> t) & 1 ? (static_cast<uint32_t>(t) * lda + lcol) * 2u : kBufOOB;
    }
#pragma unroll
    for (int q = 0; q < Sh::kPm; ++q) {
        const int r = 8 * q + sub;
        po[q] = r < k ? (static_cast<uint32_t>(r) * ldp + lcol) * 2u : kBufOOB;
    }
    auto issue = [&](int i, int stage) {   // past the band: all out of range
        const int st = first + i;
        const bool in = i < mine && st * kDmaCols + lcol < nk;
        const uint32_t dk = static_cast<uint32_t>(st * kDmaCols) * 2u;
        const uint32_t lds = ring_addr + static_cast<uint32_t>(stage * Sh::kStage);
#pragma unroll
        for (int q = 0; q < Sh::kX; ++q) {
            if constexpr (KT <= kDmaNtMaxKT) copy_to_lds_nt(ra, in ? xo[q] + dk : kBufOOB, lds + q * 1024);
            else copy_to_lds(ra, in ? xo[q] + dk : kBufOOB, lds + q * 1024);
        }
#pragma unroll
        for (int m2 = 0; m2 < S; ++m2)
#pragma unroll
            for (int q = 0; q < Sh::kPm; ++q)
                copy_to_lds(rp[m2], in ? po[q] + dk : kBufOOB, lds + (Sh::kX + m2 * Sh::kPm + q) * 1024);
    };
#pragma unroll
    for (int i = 0; i < NS - 1; ++i) issue(i, i);
    const int row = lane & 15, kg = lane >> 4;
    for (int i = 0; i < mine; ++i) {
        issue(i + NS - 1, (i + NS - 1) % NS);
        asm volatile("s_waitcnt vmcnt(%0)" :: "n"((NS - 1) * Sh::kCopies) : "memory");
        const uint8_t *base = ring + (i % NS) * Sh::kStage;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int c = 4 * h + kg;
            bf16x8 xf[MB], pf[S * KT];
#pragma unroll
            for (int m = 0; m < MB; ++m) {
                const int t = 16 * m + row;
                xf[m] = as_bf16x8(*reinterpret_cast<const u32x4 *>(base + t * 128 + ((c ^ (t & 7)) << 4)));
            }
#pragma unroll
            for (int m2 = 0; m2 < S; ++m2)
#pragma unroll
                for (int j = 0; j < KT; ++j) {
                    const int r = 16 * j + row;
                    pf[m2 * KT + j] = as_bf16x8(*reinterpret_cast<const u32x4 *>(
                        base + (Sh::kX + m2 * Sh::kPm) * 1024 + r * 128 + ((c ^ (r & 7)) << 4)));
                }
#pragma unroll
            for (int m = 0; m < MB; ++m)
#pragma unroll
                for (int j = 0; j < S * KT; ++j) acc[m][j] = mfma16_bf16(xf[m], pf[j], acc[m][j]);
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the ring is idle when the item ends
}

// A load at a uniform address of data that an earlier launch wrote and this
// kernel only reads: through the scalar cache.
template <typename T>
__device__ __forceinline__ T load_uniform(const T *p) {
    return *(const __attribute__((address_space(4))) T *)p;
}

// Valid tokens of tile `tile` of example b as a 64-bit set (bit i = token
// 64 tile + i): the listed set when the tiles were listed, else the tokens
// before T.
__device__ __forceinline__ uint64_t tile_valid(const ProjArgs &a, int j, int tile) {
    if (a.tiles) return load_uniform(a.bits + j);
    const int n = a.T - tile * TT;
    return n >= 64 ? ~0ull : (1ull << n) - 1;
}

// One chunk item (see the file comment).  Every listed tile (and, without a
// mask, every tile) has at least one valid token.  An x-side item of a layer
// whose x is shared produces the x' partials of every layer sharing it
// (S >= share_n).  The item's indices are uniform across the workgroup.
// With `ahead`, `claim` is thread 0's pending claim of the next item; after
// the last fold barrier, before any store, every wave reads it (so that the
// wait for it never waits for stores), and thread 0 publishes it in `next`.
template <int KT, int S, typename TIn>
__device__ __forceinline__ void chunk_item(const ProjArgs &a, int item, int count, f32x4 *slot, int lane,
                                           int wave, uint8_t *ring, uint32_t ring_addr, bool ahead, int claim,
                                           int *next) {
    const int rank = item / count;              // position of the work slot in processing order
    const int j = item - rank * count;          // listed tile
    int gslot = rank, l = 0;                    // work slot over all layers, and its layer
    if (a.ordered) {   // whole dwords of the argument block: scalar loads
        const uint32_t e = reinterpret_cast<const uint32_t *>(a.slot_order)[rank >> 1] >> (16 * (rank & 1));
        gslot = e & 0x3ff;
        l = (e >> 10) & 0x3f;
    } else {
        while (l + 1 < a.n_layers && gslot >= a.layer[l + 1].slot_begin) ++l;
    }
    const ChunkLayer &L = a.layer[l];
    const int cs = gslot - L.slot_begin;        // work slot of the layer: x items, then dy chunks
    const int bt = a.tiles ? load_uniform(a.tiles + j) : j;
    const int b = bt / a.tpe, tile = bt - b * a.tpe;
    const uint64_t valid = tile_valid(a, j, tile);
    constexpr bool kDma = use_dma<KT, S, TIn>();
    if constexpr (!kDma) __syncthreads();   // the previous item's reads of `slot` are done

    const bool xside = cs < L.x_items;
    const int c = xside ? cs : cs - L.x_items;
    const int n = xside ? L.n_in : L.n_out;
    const int k = xside ? a.k_in : a.k_out;
    const int nmem = xside ? L.share_n : 1;
    const int col0 = c * a.ck;
    const int nk = min(a.ck, n - col0);
    const size_t tok0 = static_cast<size_t>(b) * a.T + static_cast<size_t>(tile) * TT;
    const TIn *A = static_cast<const TIn *>(xside ? L.x : L.dy) + tok0 * n + col0;
    const TIn *P[S];
#pragma unroll
    for (int q = 0; q < S; ++q) {
        const void *pm = q >= nmem ? nullptr : xside ? a.layer[L.share[q]].p_in : L.p_out;
        P[q] = pm ? static_cast<const TIn *>(pm) + col0 : nullptr;
    }
    auto member_dst = [&](int q) {   // member q's partial slot; element (m, jj) at [(m KT + jj) 64 + lane]
        const ChunkLayer &M = xside ? a.layer[L.share[q]] : L;
        const int pslot = xside ? c : M.c_in + c;
        return reinterpret_cast<f32x4 *>(part_of(a.part, M) +
                                         (static_cast<size_t>(bt) * (M.c_in + M.c_out) + pslot) * (TT * 16 * KT)) +
               lane;
    };
    auto publish = [&]() {   // the read is unconditional, so that no path leaves the claim pending
        const int claimed = __builtin_amdgcn_readfirstlane(claim);
        if (ahead && threadIdx.x == 0) *next = static_cast<int>(gridDim.x) + claimed;
    };

    f32x4 acc[MB][S * KT];
    if constexpr (kDma) {
        const bf16_bits *Pb[S];
#pragma unroll
        for (int q = 0; q < S; ++q) Pb[q] = reinterpret_cast<const bf16_bits *>(P[q]);
        project_part_dma<KT, S>(acc, reinterpret_cast<const bf16_bits *>(A), n, Pb, n, nk, k, valid, wave, lane,
                                ring, ring_addr);
        // Waves 1..3 park their results in their own (now idle) ring; after
        // one barrier wave 0 forms ((w3 + w2) + w1) + w0 and writes it.
        constexpr int kWaveRing = DmaShape<KT, S>::kWaveRing;
        if (wave > 0) {
            f32x4 *park = reinterpret_cast<f32x4 *>(ring) + lane;
#pragma unroll
            for (int m = 0; m < MB; ++m)
#pragma unroll
                for (int jj = 0; jj < S * KT; ++jj) park[(m * S * KT + jj) * kWave] = acc[m][jj];
        }
        __syncthreads();
        publish();
        if (wave == 0) {
            const f32x4 *w1 = reinterpret_cast<const f32x4 *>(ring + kWaveRing) + lane;
            const f32x4 *w2 = reinterpret_cast<const f32x4 *>(ring + 2 * kWaveRing) + lane;
            const f32x4 *w3 = reinterpret_cast<const f32x4 *>(ring + 3 * kWaveRing) + lane;
            static_assert(NW == 4, "the fold names waves 1..3");
#pragma unroll
            for (int q = 0; q < S; ++q) {
                if (q >= nmem) break;
                f32x4 *dst = member_dst(q);
#pragma unroll
                for (int m = 0; m < MB; ++m)
#pragma unroll
                    for (int jj = 0; jj < KT; ++jj) {
                        const int e = (m * S * KT + q * KT + jj) * kWave;
                        dst[(m * KT + jj) * kWave] = ((w3[e] + w2[e]) + w1[e]) + acc[m][q * KT + jj];
                    }
            }
        }
    } else {
        bool tok_ok[MB];
#pragma unroll
        for (int m = 0; m < MB; ++m) tok_ok[m] = (valid >> (16 * m + (lane & 15))) & 1;
        project_part<KT, S, TIn, stages_for(KT)>(acc, A, n, P, n, nk, k, tok_ok, wave, lane);
        // fold the waves in the order ((w3 + w2) + w1) + w0 through `slot`
        f32x4 *my = slot + lane;
        if (wave == NW - 1) {
#pragma unroll
            for (int m = 0; m < MB; ++m)
#pragma unroll
                for (int jj = 0; jj < S * KT; ++jj) my[(m * S * KT + jj) * kWave] = acc[m][jj];
        }
        __syncthreads();
#pragma unroll
        for (int w = NW - 2; w >= 1; --w) {
            if (wave == w) {
#pragma unroll
                for (int m = 0; m < MB; ++m)
#pragma unroll
                    for (int jj = 0; jj < S * KT; ++jj)
                        my[(m * S * KT + jj) * kWave] = my[(m * S * KT + jj) * kWave] + acc[m][jj];
            }
            __syncthreads();
        }
        publish();
        if (wave == 0) {
#pragma unroll
            for (int q = 0; q < S; ++q) {
                if (q >= nmem) break;
                f32x4 *dst = member_dst(q);
#pragma unroll
                for (int m = 0; m < MB; ++m)
#pragma unroll
                    for (int jj = 0; jj < KT; ++jj)
                        dst[(m * KT + jj) * kWave] = my[(m * S * KT + q * KT + jj) * kWave] + acc[m][q * KT + jj];
            }
        }
    }
}

// Persistent: the grid is sized to the resident capacity of the GPU.  Each
// workgroup starts on item blockIdx.x and takes further items from the work
// counter.  While more than kAheadRounds rounds of items (one per
// workgroup) lie beyond its current item, it claims the next one when it
// starts the current one, so the counter's round trip overlaps the stream;
// in the last rounds it claims only when free, which keeps the tail short.  The loop
// ends once a claim passes the item count, which every workgroup reaches.
// One barrier per item hands the claim to the workgroup; the next write of
// `next` comes after the following item's fold barrier, by which time every
// thread has read it.
template <int KT, int S, typename TIn>
__global__ __launch_bounds__(NT, 1) void k_project_chunks(ProjArgs a) {
    constexpr bool kDma = use_dma<KT, S, TIn>();
    __shared__ f32x4 slot[kDma ? 1 : MB * S * KT * kWave];   // cross-wave fold of the register path
    __shared__ __attribute__((aligned(16))) uint8_t ring[kDma ? DmaShape<KT, S>::kRing : 16];
    __shared__ int next;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    constexpr int kWaveRing = kDma ? DmaShape<KT, S>::kWaveRing : 0;
    uint8_t *my_ring = ring + wave * kWaveRing;   // this wave's stages
    const int count = a.tiles ? load_uniform(a.n_tiles) : a.B * a.tpe;
    const int items = count * a.slots;
    int item = blockIdx.x;
    while (item < items) {
        const bool ahead = item + kAheadRounds * static_cast<int>(gridDim.x) < items;
        int claim = 0;
        if (ahead && tid == 0) claim = atomicAdd(a.work, 1);
        chunk_item<KT, S, TIn>(a, item, count, slot, lane, wave, my_ring, lds_addr(my_ring), ahead, claim, &next);
        if (!ahead) {
            int late = 0;
            if (tid == 0) late = atomicAdd(a.work, 1);
            late = __builtin_amdgcn_readfirstlane(late);   // waited for in every wave
            if (tid == 0) next = static_cast<int>(gridDim.x) + late;
        }
        __syncthreads();
        item = __builtin_amdgcn_readfirstlane(next);
    }
}

// ---------------------------------------------------------------------------
// k <= 16 (KT = 1), bf16 inputs that no two layers share: the per-wave stream
// of k_project_chunks, with each wave's ring kept busy from one item to the
// next.  When every layer side is one chunk (always, up to 14,336 columns) the
// items come in pairs, a tile's x side then its dy side, both in the same
// workgroup: the writer keeps the folded x' in registers and, after the dy
// fold, forms the tile's 16 x 16 sum with the MFMAs of k_project_tile_finish<1>
// (same operands, same order, so the same bits) straight into gpart.  No chunk
// partial is written and the tile-sum kernel is not launched; the example sums
// skip the tiles without a valid token, whose sums were never written.
//
// In k_project_chunks every item starts with an empty ring and ends with a
// drained one, so each item pays a memory latency before its first step.  At
// 768 to 4,096 columns per layer side an item is 3 to 24 steps per wave, and
// that latency is a large share of it.  Here the ring runs on: during the
// last two steps of an item a wave issues the copies of the first two steps of
// its band of the next item.  For that the next item must be known when an
// item starts, so items are claimed two ahead (the first two of a workgroup
// are blockIdx.x and blockIdx.x + gridDim.x).  A fifth wave does everything
// besides the streaming: it claims the items, decodes each (its layer, tile,
// operands, valid-token set and partial slot: a chain of dependent loads that
// took a streaming wave about 1,800 cycles per item) and publishes it through
// LDS, and it folds the four waves' partials, parked in one of two LDS buffers at
// each item's end, in the order of k_project_chunks, ((w3 + w2) + w1) + w0,
// and writes them.  The streaming waves issue no memory operation but their
// copies, so "at most the two later steps' copies pending" is an exact wait,
// and one barrier per item (LDS operations only) hands over the partials and
// the next claim.  A band shorter than two steps is padded with empty steps
// (out-of-range copies, no products) so that the look-ahead never passes the
// next item.  Each wave's band, step order and sums are those of
// k_project_chunks, so the results are the same bits.
constexpr int kStreamNT = (NW + 1) * kWave;   // four streaming waves and the writer
using StreamSh = DmaShape<1, 1>;
constexpr int kStreamNS = StreamSh::kStages;
static_assert(kStreamNS == 3, "the look-ahead is two steps");

// An unshared item's operands and partial slot (the fields chunk_item uses
// with S = 1).
struct StreamItem {
    const bf16_bits *A, *P;
    int n, k, nk;
    uint64_t valid;
    size_t dst;   // float offset of the chunk partial in a.part
};

__device__ __forceinline__ StreamItem stream_item(const ProjArgs &a, int item, int count) {
    const int unit = a.paired ? item >> 1 : item;   // a pair or an item
    const int rank = unit / count;
    const int j = unit - rank * count;
    int gslot = rank, l = 0;
    if (a.ordered) {
        const uint32_t e = reinterpret_cast<const uint32_t *>(a.slot_order)[rank >> 1] >> (16 * (rank & 1));
        gslot = (e & 0x3ff) + (a.paired ? item & 1 : 0);
        l = (e >> 10) & 0x3f;
    } else {
        while (l + 1 < a.n_layers && gslot >= a.layer[l + 1].slot_begin) ++l;
    }
    // the layer table is indexed by integers (no selects or phis of pointers into
    // the kernel arguments, which would keep them in a private copy)
    const int cs = gslot - a.layer[l].slot_begin;
    const int bt = a.tiles ? load_uniform(a.tiles + j) : j;
    const int b = bt / a.tpe, tile = bt - b * a.tpe;
    const bool xside = cs < a.layer[l].x_items;
    const int c = xside ? cs : cs - a.layer[l].x_items;
    const int m = xside ? a.layer[l].share[0] : l;   // the layer whose partial slots hold the item
    StreamItem it;
    it.valid = tile_valid(a, j, tile);
    it.n = xside ? a.layer[l].n_in : a.layer[l].n_out;
    it.k = xside ? a.k_in : a.k_out;
    const int col0 = c * a.ck;
    it.nk = min(a.ck, it.n - col0);
    const size_t tok0 = static_cast<size_t>(b) * a.T + static_cast<size_t>(tile) * TT;
    const void *src = xside ? a.layer[l].x : a.layer[l].dy;
    const void *proj = xside ? a.layer[m].p_in : a.layer[l].p_out;
    it.A = static_cast<const bf16_bits *>(src) + tok0 * it.n + col0;
    it.P = static_cast<const bf16_bits *>(proj) + col0;
    const int c_in = a.layer[m].c_in, c_out = a.layer[m].c_out;
    const int pslot = xside ? c : c_in + c;
    // paired: the tile's 16 x 16 sum in gpart; else the chunk partial in part
    it.dst = a.paired ? (static_cast<size_t>(l) * a.B * a.tpe + bt) * 256
                      : static_cast<size_t>(a.layer[m].part_unit) * kPartUnit +
                            (static_cast<size_t>(bt) * (c_in + c_out) + pslot) * (TT * 16);
    return it;
}

// One streaming wave's band of an item: steps first .. first + mine - 1 of
// the chunk, padded to len >= kStreamNS - 1 steps.
struct StreamBand {
    __amdgpu_buffer_rsrc_t ra, rp;
    uint32_t xo[StreamSh::kX], po[StreamSh::kPm];
    int first, mine, len, nk;
};

__device__ __forceinline__ void stream_band(StreamBand &d, const StreamItem &it, int wave, int sub, int lcol) {
    const int nsteps = (it.nk + kDmaCols - 1) / kDmaCols;
    const int per = (nsteps + NW - 1) / NW;
    d.first = wave * per;
    d.mine = max(0, min(per, nsteps - d.first));
    d.len = max(d.mine, kStreamNS - 1);
    d.nk = it.nk;
    d.ra = buf_rsrc(it.A, (static_cast<uint32_t>(TT - 1) * it.n + it.nk) * 2u);
    d.rp = buf_rsrc(it.P, (static_cast<uint32_t>(it.k - 1) * it.n + it.nk) * 2u);
#pragma unroll
    for (int q = 0; q < StreamSh::kX; ++q) {
        const int t = 8 * q + sub;
        d.xo[q] = (it.valid >> t) & 1 ? (static_cast<uint32_t>(t) * it.n + lcol) * 2u : kBufOOB;
    }
#pragma unroll
    for (int q = 0; q < StreamSh::kPm; ++q) {
        const int r = 8 * q + sub;
        d.po[q] = r < it.k ? (static_cast<uint32_t>(r) * it.n + lcol) * 2u : kBufOOB;
    }
}

// A decoded item as the writer wave publishes it in LDS: 12 words (A, P,
// valid, dst as low / high halves, then n, k, nk) at the start of a 64-word
// slot.  Lane l writes word l, the lanes past 12 write padding, so the store
// needs no branch on the lane (a divergent branch around the decode would
// move the kernel arguments it indexes into scratch memory).
constexpr int kItemWords = 12;
typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
// (The slot pointers carry the LDS address space: through generic pointers
// the accesses might alias private memory, and the kernel arguments would be
// kept in a private copy.)
__device__ __forceinline__ void item_to_lds(lds_u32 *slot, const StreamItem &it, int lane) {
    const uint64_t A = reinterpret_cast<uintptr_t>(it.A), P = reinterpret_cast<uintptr_t>(it.P);
    const uint64_t dst = static_cast<uint64_t>(it.dst);
    const uint32_t w[kItemWords] = {static_cast<uint32_t>(A),         static_cast<uint32_t>(A >> 32),
                                    static_cast<uint32_t>(P),         static_cast<uint32_t>(P >> 32),
                                    static_cast<uint32_t>(it.valid),  static_cast<uint32_t>(it.valid >> 32),
                                    static_cast<uint32_t>(dst),       static_cast<uint32_t>(dst >> 32),
                                    static_cast<uint32_t>(it.n),      static_cast<uint32_t>(it.k),
                                    static_cast<uint32_t>(it.nk),     0u};
    uint32_t v = 0;
#pragma unroll
    for (int q = 0; q < kItemWords; ++q) v = lane == q ? w[q] : v;
    slot[lane] = v;
}

// The read-back: every lane reads the same words, made wave-uniform.
__device__ __forceinline__ StreamItem item_from_lds(const lds_u32 *slot) {
    const u32x4 q0 = reinterpret_cast<const lds_u32x4 *>(slot)[0];
    const u32x4 q1 = reinterpret_cast<const lds_u32x4 *>(slot)[1];
    const u32x4 q2 = reinterpret_cast<const lds_u32x4 *>(slot)[2];
    auto u = [](uint32_t v) { return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(v))); };
    auto u64 = [&](uint32_t lo, uint32_t hi) { return static_cast<uint64_t>(u(lo)) | static_cast<uint64_t>(u(hi)) << 32; };
    StreamItem it;
    it.A = reinterpret_cast<const bf16_bits *>(static_cast<uintptr_t>(u64(q0[0], q0[1])));
    it.P = reinterpret_cast<const bf16_bits *>(static_cast<uintptr_t>(u64(q0[2], q0[3])));
    it.valid = u64(q1[0], q1[1]);
    it.dst = static_cast<size_t>(u64(q1[2], q1[3]));
    it.n = static_cast<int>(u(q2[0]));
    it.k = static_cast<int>(u(q2[1]));
    it.nk = static_cast<int>(u(q2[2]));
    return it;
}

// The band of no item (past the last): every copy out of range.
__device__ __forceinline__ void stream_band_none(StreamBand &d, const bf16_bits *base) {
    d.first = 0;
    d.mine = 0;
    d.len = kStreamNS - 1;
    d.nk = 0;
    d.ra = buf_rsrc(base, 0u);
    d.rp = buf_rsrc(base, 0u);
#pragma unroll
    for (int q = 0; q < StreamSh::kX; ++q) d.xo[q] = kBufOOB;
#pragma unroll
    for (int q = 0; q < StreamSh::kPm; ++q) d.po[q] = kBufOOB;
}

// Copies of band position p into the stage at LDS address lds (as the issue of
// project_part_dma).
__device__ __forceinline__ void stream_issue(const StreamBand &d, int p, uint32_t lds, int lcol) {
    const int st = d.first + p;
    const bool in = p < d.mine && st * kDmaCols + lcol < d.nk;
    const uint32_t dk = static_cast<uint32_t>(st * kDmaCols) * 2u;
#pragma unroll
    for (int q = 0; q < StreamSh::kX; ++q) copy_to_lds_nt(d.ra, in ? d.xo[q] + dk : kBufOOB, lds + q * 1024);
#pragma unroll
    for (int q = 0; q < StreamSh::kPm; ++q)
        copy_to_lds(d.rp, in ? d.po[q] + dk : kBufOOB, lds + (StreamSh::kX + q) * 1024);
}

// The products of one step (as project_part_dma).
__device__ __forceinline__ void stream_step(f32x4 (&acc)[MB], const uint8_t *base, int lane) {
    const int row = lane & 15, kg = lane >> 4;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int c = 4 * h + kg;
        bf16x8 xf[MB];
#pragma unroll
        for (int m = 0; m < MB; ++m) {
            const int t = 16 * m + row;
            xf[m] = as_bf16x8(*reinterpret_cast<const u32x4 *>(base + t * 128 + ((c ^ (t & 7)) << 4)));
        }
        const bf16x8 pf =
            as_bf16x8(*reinterpret_cast<const u32x4 *>(base + StreamSh::kX * 1024 + row * 128 + ((c ^ (row & 7)) << 4)));
#pragma unroll
        for (int m = 0; m < MB; ++m) acc[m] = mfma16_bf16(xf[m], pf, acc[m]);
    }
}

// LDS writes done, then the workgroup barrier; no wait for copies in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__global__ __launch_bounds__(kStreamNT, 1) void k_project_stream(ProjArgs a) {
    constexpr int NS = kStreamNS;
    __shared__ __attribute__((aligned(16))) uint8_t ring[StreamSh::kRing];
    __shared__ f32x4 fold[2][NW][MB * kWave];
    __shared__ int queue[4];
    __shared__ __attribute__((aligned(16))) uint32_t decoded[4][kWave];   // the claimed items, decoded (slots of queue)
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave);
    const int count = a.tiles ? load_uniform(a.n_tiles) : a.B * a.tpe;
    const int items = count * a.slots;
    const int grid = static_cast<int>(gridDim.x);
    // the first two items: pair blockIdx.x (paired), else items blockIdx.x and blockIdx.x + gridDim.x
    int cur = a.paired ? 2 * static_cast<int>(blockIdx.x) : static_cast<int>(blockIdx.x);
    int nxt = a.paired ? cur + 1 : cur + grid;

    if (wave == NW) {   // the writer: claims, decodes, publishes, folds and writes
        f32x4 xk[MB];   // paired: the x' of the pair being formed
        auto fold_out = [&](int item, size_t dst, const f32x4 (*w)[MB * kWave]) {
            f32x4 v[MB];
#pragma unroll
            for (int m = 0; m < MB; ++m) {
                const int e = m * kWave + lane;
                v[m] = ((w[3][e] + w[2][e]) + w[1][e]) + w[0][e];
            }
            if (!a.paired) {
                f32x4 *d = reinterpret_cast<f32x4 *>(a.part + dst) + lane;
#pragma unroll
                for (int m = 0; m < MB; ++m) d[m * kWave] = v[m];
            } else if ((item & 1) == 0) {
#pragma unroll
                for (int m = 0; m < MB; ++m) xk[m] = v[m];
            } else {   // the tile's sum, as k_project_tile_finish<1> forms it from the partials
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int m = 0; m < MB; ++m) {
                    const f32x4 dv = f32x4{0.f, 0.f, 0.f, 0.f} + v[m], xv = f32x4{0.f, 0.f, 0.f, 0.f} + xk[m];
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc = mfma16_f32(dv[r], xv[r], acc);
                }
                float *g = a.gpart + dst + lane;
#pragma unroll
                for (int r = 0; r < 4; ++r) g[64 * r] = acc[r];
            }
        };
        // output offsets of the items in flight: prev (folded now), cur, nxt
        size_t part_prev = 0, part_cur = cur < items ? stream_item(a, cur, count).dst : 0;
        size_t part_nxt = nxt < items ? stream_item(a, nxt, count).dst : 0;
        int prev = -1;
        int n = 0;
        for (; cur < items; ++n) {
            int claim = items;   // none (any value >= items)
            size_t part_claim = 0;
            if (nxt < items) {
                if (a.paired && (n & 1)) {
                    claim = nxt + 1;   // the dy side of the pair whose x side (nxt) is at position n + 1
                } else {   // a new pair (paired: position n + 2 is even) or a new item
                    int c = 0;
                    if (lane == 0) c = atomicAdd(a.work, 1);
                    c = __builtin_amdgcn_readfirstlane(c);
                    claim = a.paired ? 2 * (grid + c) : 2 * grid + c;
                }
            }
            if (lane == 0) queue[(n + 2) & 3] = claim;
            if (claim < items) {   // the streaming waves take it decoded
                const StreamItem it = stream_item(a, claim, count);
                part_claim = it.dst;
                item_to_lds((lds_u32 *)decoded[(n + 2) & 3], it, lane);
            }
            if (prev >= 0) fold_out(prev, part_prev, fold[(n - 1) & 1]);
            lds_barrier();   // B_n: the partials of item n are parked, item n + 2 is published
            prev = cur;
            part_prev = part_cur;
            cur = nxt;
            part_cur = part_nxt;
            nxt = claim;
            part_nxt = part_claim;
        }
        if (prev >= 0) fold_out(prev, part_prev, fold[(n - 1) & 1]);
        return;
    }

    // streaming waves
    const int sub = lane >> 3;
    const int lcol = ((lane & 7) ^ sub) * 8;   // the lane's element column within a step
    uint8_t *my_ring = ring + wave * StreamSh::kWaveRing;
    const uint32_t ring_addr = lds_addr(my_ring);
    StreamBand dc, dn;
    int iss = 0, con = 0;   // stages of the next copy and of the next step
    if (cur < items) {
        stream_band(dc, stream_item(a, cur, count), wave, sub, lcol);
#pragma unroll
        for (int p = 0; p < NS - 1; ++p) {
            stream_issue(dc, p, ring_addr + iss * StreamSh::kStage, lcol);
            iss = iss == NS - 1 ? 0 : iss + 1;
        }
    }
    // item 1 of the workgroup is decoded here; the later ones, claimed, come decoded from the writer
    if (nxt < items) stream_band(dn, stream_item(a, nxt, count), wave, sub, lcol);
    else stream_band_none(dn, static_cast<const bf16_bits *>(a.layer[0].x));
    for (int n = 0; cur < items; ++n) {
        if (n > 0) {
            if (nxt < items) stream_band(dn, item_from_lds((const lds_u32 *)decoded[(n + 1) & 3]), wave, sub, lcol);
            else stream_band_none(dn, static_cast<const bf16_bits *>(a.layer[0].x));
        }
        f32x4 acc[MB];
#pragma unroll
        for (int m = 0; m < MB; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int p = 0; p < dc.len; ++p) {
            const int q = p + NS - 1;   // the position two steps ahead, in this item or the next
            const uint32_t lds = ring_addr + iss * StreamSh::kStage;
            if (q < dc.len) stream_issue(dc, q, lds, lcol);
            else stream_issue(dn, q - dc.len, lds, lcol);
            iss = iss == NS - 1 ? 0 : iss + 1;
            // the copies of position p are done when only the two later positions' are pending
            asm volatile("s_waitcnt vmcnt(%0)" :: "n"((NS - 1) * StreamSh::kCopies) : "memory");
            if (p < dc.mine) stream_step(acc, my_ring + con * StreamSh::kStage, lane);
            con = con == NS - 1 ? 0 : con + 1;
        }
        f32x4 *park = fold[n & 1][wave] + lane;
#pragma unroll
        for (int m = 0; m < MB; ++m) park[m * kWave] = acc[m];
        lds_barrier();   // B_n
        const int after = __builtin_amdgcn_readfirstlane(queue[(n + 2) & 3]);
        cur = nxt;
        nxt = after;
        dc = dn;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the copies issued for no item
}

// ---------------------------------------------------------------------------
// bf16, unshared inputs: tile groups sharing one projection slab.
//
// At k = 64 a P slab (64 rows x 128 B per 64-column step) is as large as a
// 64-token x slab, so a ring stage per wave holding both leaves room for only
// two stages in LDS: about 32 KB of HBM reads in flight per CU.  Here a work
// item is one contraction chunk of one side of one layer for a GROUP of up
// to four listed tiles: wave w streams tile w of the group over all of the
// chunk's 64-column steps, and the four waves share each step's P slab (each
// wave copies its share of it).  A stage is four x slabs and one P slab
// (34 KB at k <= 16, 36 KB at k <= 32, 40 KB at k <= 64, 48 KB at k <= 128), so
// four stages fit at k <= 32 and three above, all but one in flight.  One
// barrier per step makes every wave's share of the P slab visible and frees
// the stage the next copies overwrite.  Each wave sums its tile over the
// whole chunk, so no cross-wave fold is needed; the tile's partial goes to
// the workspace in the same layout as the per-wave path's.  In paired units
// (16 < k <= 64, every layer side one chunk) a workgroup takes a group's x
// item and then its dy item, and each wave forms its tile's sum from the two
// (the 7-layer block at k = 64: 494 -> 452 us).
//
// Two measured choices keep the HBM stream fast.  The x / dy copies carry the
// non-temporal hint (the projection slabs, re-read by every group, keep the
// cache).  And each group walks the chunk's steps from its own starting
// step, 37 x group mod steps, so that the groups streaming one chunk at the
// same time on all CUs read scattered column ranges rather than the same
// columns of different rows (starts spaced evenly, group x steps / groups,
// keep groups that run side by side on nearby columns and measured 4% slower).
// The 7-layer block at k = 64 (B = 16, T = 1024): 570 us with the per-wave
// path, 581 with tile groups alone, 549 with the scattered start, 559 with the
// hint, 494-497 with both.
template <int KT>
struct TileDma {
    static constexpr int kX = TT / 8;                    // x slab: 8 copies of 8 token rows
    static constexpr int kP = 2 * KT;                    // P slab: 16 KT rows, 8 per copy
    static constexpr int kPw = (kP + NW - 1) / NW;       // P copies issued by each wave (at most)
    static constexpr int kCopies = kX + kPw;             // copies per wave per stage (at most)
    static constexpr int kStage = (NW * kX + kP) * 1024; // bytes of one stage
    static constexpr int kStages = 4 * kStage + 1024 <= 160 * 1024 ? 4 : 3;
    static constexpr int kRing = kStages * kStage;
    static_assert(kRing + 1024 <= 160 * 1024, "the ring fits in LDS");
};

// Wait until at most kCount of this wave's copies are pending (its copies of
// the later stages), then meet the other waves at the barrier.
template <int kCount>
__device__ __forceinline__ void wait_copies_below() {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(kCount) : "memory");
}

// Paired units in the tile-group kernel up to KT = 4 (at KT = 8 the kept x
// side would be 128 more registers per lane).
constexpr int kMaxPairedKT = 4;
template <int KT>
constexpr bool kTilePairs = KT <= kMaxPairedKT;

// What a tile-group item does with each wave's projection of its tile:
// write it as the chunk partial (the tile-sum kernel reads it), keep it in
// registers (the x side of a paired unit), or form the tile's sum from it
// (the dy side) and the kept x side.
enum TileFold { kFoldPart, kFoldKeepX, kFoldTileSum };

template <int KT, TileFold F>
__device__ __forceinline__ void tile_group_item(const ProjArgs &a, int item, int count, int groups, int lane,
                                                int wave, uint32_t ring_addr, const uint8_t *ring,
                                                f32x4 (&xk)[MB][KT]) {
    using Sh = TileDma<KT>;
    constexpr int NS = Sh::kStages;
    // paired: item 2 u is unit u's x side, item 2 u + 1 its dy side (the layer's
    // x slot and the slot after it, one chunk each)
    const int unit = F == kFoldPart ? item : item >> 1;
    const int side = F == kFoldPart ? 0 : item & 1;
    const int rank = unit / groups;             // position of the work slot (paired: layer) in processing order
    const int grp = unit - rank * groups;       // group of listed tiles
    int gslot = rank, l = 0;
    if (a.ordered) {
        const uint32_t e = reinterpret_cast<const uint32_t *>(a.slot_order)[rank >> 1] >> (16 * (rank & 1));
        gslot = (e & 0x3ff) + side;
        l = (e >> 10) & 0x3f;
    } else {
        while (l + 1 < a.n_layers && gslot >= a.layer[l + 1].slot_begin) ++l;
    }
    const ChunkLayer &L = a.layer[l];
    const int cs = gslot - L.slot_begin;        // x chunks first, then dy chunks
    const bool xside = cs < L.x_items;
    const int c = xside ? cs : cs - L.x_items;
    const int n = xside ? L.n_in : L.n_out;
    const int k = xside ? a.k_in : a.k_out;
    const int col0 = c * a.ck;
    const int nk = min(a.ck, n - col0);
    // this wave's tile
    const int j = grp * NW + wave;
    const bool has = j < count;
    int bt = 0;
    uint64_t valid = 0;
    if (has) {
        bt = a.tiles ? load_uniform(a.tiles + j) : j;
        valid = tile_valid(a, j, bt - (bt / a.tpe) * a.tpe);
    }
    const int b = bt / a.tpe, tile = bt - b * a.tpe;
    const size_t tok0 = static_cast<size_t>(b) * a.T + static_cast<size_t>(tile) * TT;
    const bf16_bits *A = static_cast<const bf16_bits *>(xside ? L.x : L.dy) + tok0 * n + col0;
    const bf16_bits *Pm = static_cast<const bf16_bits *>(xside ? L.p_in : L.p_out) + col0;
    const auto ra = buf_rsrc(A, has ? (static_cast<uint32_t>(TT - 1) * n + nk) * 2u : 0u);
    const auto rp = buf_rsrc(Pm, (static_cast<uint32_t>(k - 1) * n + nk) * 2u);
    const int sub = lane >> 3;
    const int lcol = ((lane & 7) ^ sub) * 8;     // the lane's element column within a step
    // P copies of this wave: kPw, or fewer where the slab has fewer than NW kPw copies
    constexpr bool kEven = Sh::kPw * NW == Sh::kP;
    const int pw = kEven ? Sh::kPw : (wave * Sh::kPw < Sh::kP ? Sh::kPw : 0);
    uint32_t xo[Sh::kX], po[Sh::kPw];
#pragma unroll
    for (int q = 0; q < Sh::kX; ++q) {
        const int t = 8 * q + sub;
        xo[q] = (valid >> t) & 1 ? (static_cast<uint32_t>(t) * n + lcol) * 2u : kBufOOB;
    }
#pragma unroll
    for (int q = 0; q < Sh::kPw; ++q) {
        const int r = 8 * (wave * Sh::kPw + q) + sub;
        po[q] = r < k ? (static_cast<uint32_t>(r) * n + lcol) * 2u : kBufOOB;
    }
    const int nsteps = (nk + kDmaCols - 1) / kDmaCols;
    const int rot = (grp * 37) % nsteps;   // the group's first step: scattered over the chunk
    // stage layout: x slab of wave 0..3 (8 KB each), then the P slab
    auto issue = [&](int st, int stage) {   // steps past the chunk's count: all out of range
        int sr = st + rot;
        if (sr >= nsteps) sr -= nsteps;
        const bool in = st < nsteps && sr * kDmaCols + lcol < nk;
        const uint32_t dk = static_cast<uint32_t>(sr * kDmaCols) * 2u;
        const uint32_t lds = ring_addr + static_cast<uint32_t>(stage * Sh::kStage);
#pragma unroll
        for (int q = 0; q < Sh::kX; ++q)
            copy_to_lds_nt(ra, in ? xo[q] + dk : kBufOOB, lds + (wave * Sh::kX + q) * 1024);
#pragma unroll
        for (int q = 0; q < Sh::kPw; ++q)
            if (kEven || pw > 0)
                copy_to_lds(rp, in ? po[q] + dk : kBufOOB, lds + (NW * Sh::kX + wave * Sh::kPw + q) * 1024);
    };
    f32x4 acc[MB][KT];
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int jj = 0; jj < KT; ++jj) acc[m][jj] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < NS - 1; ++i) issue(i, i);
    const int row = lane & 15, kg = lane >> 4;
    for (int i = 0; i < nsteps; ++i) {
        // this wave's copies of step i are done when only the NS - 2 later
        // stages are pending; after the barrier every wave's are, and every
        // wave has finished reading step i - 1, whose stage the next copies refill
        if (kEven || pw > 0) wait_copies_below<(NS - 2) * Sh::kCopies>();
        else wait_copies_below<(NS - 2) * Sh::kX>();
        issue(i + NS - 1, (i + NS - 1) % NS);
        if (!has) continue;
        const uint8_t *base = ring + (i % NS) * Sh::kStage;
        const uint8_t *xb = base + wave * Sh::kX * 1024;
        const uint8_t *pbase = base + NW * Sh::kX * 1024;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int cc = 4 * h + kg;
            bf16x8 xf[MB], pf[KT];
#pragma unroll
            for (int m = 0; m < MB; ++m) {
                const int t = 16 * m + row;
                xf[m] = as_bf16x8(*reinterpret_cast<const u32x4 *>(xb + t * 128 + ((cc ^ (t & 7)) << 4)));
            }
#pragma unroll
            for (int jj = 0; jj < KT; ++jj) {
                const int r = 16 * jj + row;
                pf[jj] = as_bf16x8(*reinterpret_cast<const u32x4 *>(pbase + r * 128 + ((cc ^ (r & 7)) << 4)));
            }
#pragma unroll
            for (int m = 0; m < MB; ++m)
#pragma unroll
                for (int jj = 0; jj < KT; ++jj) acc[m][jj] = mfma16_bf16(xf[m], pf[jj], acc[m][jj]);
        }
    }
    // the copies past the chunk (out of range: zeros) are still in flight
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (!has) return;
    if constexpr (F == kFoldPart) {
        const int pslot = xside ? c : L.c_in + c;
        f32x4 *dst = reinterpret_cast<f32x4 *>(part_of(a.part, L) +
                                               (static_cast<size_t>(bt) * (L.c_in + L.c_out) + pslot) *
                                                   (TT * 16 * KT)) + lane;
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int jj = 0; jj < KT; ++jj) dst[(m * KT + jj) * kWave] = acc[m][jj];
    } else if constexpr (F == kFoldKeepX) {
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int jj = 0; jj < KT; ++jj) xk[m][jj] = acc[m][jj];
    } else {
        // The tile's sum over tokens of dy'_t x'_t^T, block (jo, ji) as the
        // tile-sum kernel forms it from the partials (which hold x' and dy' in
        // this lane layout): the same fp32 16x16x4 MFMAs in the same order,
        // on the same operands (0 + v, as its sum over one chunk gives).
        const int per_layer = a.B * a.tpe;
        float *gdst = a.gpart + static_cast<size_t>(l * per_layer + bt) * (16 * KT * 16 * KT) + lane;
#pragma unroll
        for (int jo = 0; jo < KT; ++jo)
#pragma unroll
            for (int ji = 0; ji < KT; ++ji) {
                f32x4 g = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int m = 0; m < MB; ++m)
#pragma unroll
                    for (int r = 0; r < 4; ++r) g = mfma16_f32(0.f + acc[m][jo][r], 0.f + xk[m][ji][r], g);
#pragma unroll
                for (int r = 0; r < 4; ++r) gdst[(jo * KT + ji) * 256 + 64 * r] = g[r];
            }
    }
}

// Persistent, like k_project_chunks: items are (work slot, tile group), taken
// from the work counter, claimed ahead except in the last rounds.  The
// barrier that hands a claim to the workgroup also keeps the next item's
// first copies from overwriting a stage another wave is still reading.
template <int KT, bool kPaired>
__global__ __launch_bounds__(NT, 1) void k_project_tiles(ProjArgs a) {
    __shared__ __attribute__((aligned(16))) uint8_t ring[TileDma<KT>::kRing];
    __shared__ int next;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int count = a.tiles ? load_uniform(a.n_tiles) : a.B * a.tpe;
    const int groups = (count + NW - 1) / NW;
    const int items = groups * a.slots;
    const uint32_t ring_addr = lds_addr(ring);
    f32x4 xk[MB][KT];   // paired: this wave's x side of the unit's tile
    // paired: units of two items (a tile group's x side, then its dy side)
    const int units = kPaired ? items / 2 : items;
    int u = blockIdx.x;
    while (u < units) {
        const bool ahead = u + kAheadRounds * static_cast<int>(gridDim.x) < units;
        int claim = 0;
        if (ahead && tid == 0) claim = atomicAdd(a.work, 1);
        if constexpr (kPaired) {
            tile_group_item<KT, kFoldKeepX>(a, 2 * u, count, groups, lane, wave, ring_addr, ring, xk);
            __syncthreads();   // the dy side's first copies refill stages the x side read
            tile_group_item<KT, kFoldTileSum>(a, 2 * u + 1, count, groups, lane, wave, ring_addr, ring, xk);
        } else {
            tile_group_item<KT, kFoldPart>(a, u, count, groups, lane, wave, ring_addr, ring, xk);
        }
        if (tid == 0) next = static_cast<int>(gridDim.x) + (ahead ? claim : atomicAdd(a.work, 1));
        __syncthreads();
        u = __builtin_amdgcn_readfirstlane(next);
        __syncthreads();   // every wave has read `next` before it is written again
    }
}

// Bit i set where byte i of w is non-zero (i < 4).
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t w) {
    return ((w & 0xffu) != 0) | (((w >> 8) & 0xffu) != 0) << 1 | (((w >> 16) & 0xffu) != 0) << 2 |
           ((w >> 24) != 0) << 3;
}

// Clears the work counter and, with a mask, lists the tiles that hold at
// least one valid token, in tile order, each with its set of valid tokens
// (one workgroup; block-wide prefix counts keep the order).  A full tile's
// 64 mask bytes are read as four 128-bit loads when the mask rows are
// 16-byte aligned.
__global__ __launch_bounds__(1024) void k_project_prep(const uint8_t *mask, int B, int T, int tpe, int *tiles,
                                                        uint64_t *bits, uint64_t *tile_bits, int *n_tiles,
                                                        int *work) {
    __shared__ int wsum[16];
    __shared__ int base;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) {
        *work = 0;
        base = 0;
    }
    if (mask == nullptr) return;
    const bool vec = (reinterpret_cast<uintptr_t>(mask) & 15) == 0 && (T & 15) == 0;
    __syncthreads();
    const int total = B * tpe;
    for (int t0 = 0; t0 < total; t0 += 1024) {
        const int bt = t0 + tid;
        uint64_t set = 0;
        if (bt < total) {
            const int b = bt / tpe, tile = bt - b * tpe;
            const uint8_t *m = mask + static_cast<size_t>(b) * T + static_cast<size_t>(tile) * TT;
            const int n = min(TT, T - tile * TT);
            if (vec && n == TT) {
#pragma unroll
                for (int q = 0; q < TT / 16; ++q) {
                    const u32x4 v = ld128(m + 16 * q);
#pragma unroll
                    for (int e = 0; e < 4; ++e) set |= static_cast<uint64_t>(nonzero_bytes(v[e])) << (16 * q + 4 * e);
                }
            } else {
                for (int i = 0; i < n; ++i) set |= static_cast<uint64_t>(m[i] != 0) << i;
            }
        }
        if (bt < total) tile_bits[bt] = set;
        const int any = set != 0;
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
            tiles[base + before + x - 1] = bt;
            bits[base + before + x - 1] = set;
        }
        __syncthreads();
        if (tid == 0) base += all;
        __syncthreads();
    }
    if (tid == 0) *n_tiles = base;
}

// One wave per (tile, 16 x 16 block (jo, ji) of G): x' and dy' of the tile
// are the fixed-order sums of their chunk partials, read straight from the
// workspace, where they already sit in the operand layout of the fp32
// 16x16x4 MFMA with the token as the contraction index (lane l of partial
// block (m, j) holds the rows t = 16 m + 4 (l / 16) + r, r < 4, of column
// 16 j + l % 16).  So the block of the tile's sum over tokens of dy'_t x'_t^T
// is 16 MFMAs over (m, r).  Tiles without a valid token get 0.
template <int KT>
__global__ __launch_bounds__(256) void k_project_tile_finish(ProjArgs a, int pairs) {
    constexpr int KP = 16 * KT;
    constexpr int NQ = MB * KT * kWave;     // f32x4 per chunk partial
    const int lane = threadIdx.x & (kWave - 1);
    const int p = blockIdx.x * NW + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    if (p >= pairs) return;
    const int tix = p / (KT * KT), blk = p - tix * (KT * KT);   // tile over all layers, block of G
    const int jo = blk / KT, ji = blk - jo * KT;
    const int per_layer = a.B * a.tpe;
    const int l = tix / per_layer;
    const int bt = tix - l * per_layer;
    // the tile's sum, block by block in the MFMA result layout: block (jo, ji)
    // holds register r of lane l at 256 (jo KT + ji) + 64 r + l
    float *gdst = a.gpart + static_cast<size_t>(tix) * (KP * KP) + blk * 256 + lane;
    // every tile below tpe holds a token before T; with a mask, the tile's set from
    // prep.  An empty tile's block is 0 and its partial slots (never written) are
    // not read: with ragged batches that is a third or more of the reads here.
    const bool any = a.mask == nullptr || load_uniform(a.tile_bits + bt) != 0;
    if (!any) {
#pragma unroll
        for (int r = 0; r < 4; ++r) gdst[64 * r] = 0.f;
        return;
    }
    const ChunkLayer &L = a.layer[l];
    const int C = L.c_in + L.c_out;
    const f32x4 *src = reinterpret_cast<const f32x4 *>(part_of(a.part, L) + static_cast<size_t>(bt) * C * (TT * KP)) + lane;
    f32x4 dv[MB], xv[MB];
#pragma unroll
    for (int m = 0; m < MB; ++m) dv[m] = xv[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < L.c_in; ++c)
#pragma unroll
        for (int m = 0; m < MB; ++m) xv[m] += src[static_cast<size_t>(c) * NQ + (m * KT + ji) * kWave];
    for (int c = L.c_in; c < C; ++c)
#pragma unroll
        for (int m = 0; m < MB; ++m) dv[m] += src[static_cast<size_t>(c) * NQ + (m * KT + jo) * kWave];
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc = mfma16_f32(dv[m][r], xv[m][r], acc);
    // result register r of lane l: o = 16 jo + 4 (l / 16) + r, i = 16 ji + l % 16
    // (whole 256-byte rows per store; entries past k_out or k_in are never read)
#pragma unroll
    for (int r = 0; r < 4; ++r) gdst[64 * r] = acc[r];
}

// The same sums for KT >= 2, one workgroup per tile: the tile's x' and dy'
// (the fixed-order sums of their chunk partials) are read once into LDS,
// rather than once per 16 x 16 block of G that needs them (KT times each),
// and wave w forms blocks w, w + 4, ... from there with the same MFMAs in the
// same order, so the results are those of k_project_tile_finish.
template <int KT>
__global__ __launch_bounds__(256) void k_project_tile_finish_wg(ProjArgs a) {
    constexpr int KP = 16 * KT;
    constexpr int NQ = MB * KT * kWave;     // f32x4 per chunk partial
    static_assert(NQ == 256 * KT, "thread t sums elements t + 256 u, u < KT");
    // Thread (wave w, lane) sums elements 256 u + 64 w + lane, u < KT: block row
    // 4 u + w of the partial.  From KT = 4 on, w's blocks (jo, ji) all have ji = w
    // (mod 4), so the x' it sums are the x' it needs and only dy' goes through LDS
    // (half the LDS, so one round of workgroups fits the CUs at k = 64).
    constexpr bool kOwnX = KT % 4 == 0;
    __shared__ f32x4 xs[kOwnX ? 1 : NQ], ds[NQ];
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int tix = blockIdx.x;              // tile over all layers
    const int per_layer = a.B * a.tpe;
    const int l = tix / per_layer;
    const int bt = tix - l * per_layer;
    const bool any = a.mask == nullptr || load_uniform(a.tile_bits + bt) != 0;
    float *gdst = a.gpart + static_cast<size_t>(tix) * (KP * KP) + lane;
    if (!any) {   // no valid token: the tile's sum is 0 (its partial slots were never written)
        for (int e = tid; e < KP * KP; e += 256) gdst[e - lane] = 0.f;
        return;
    }
    const ChunkLayer &L = a.layer[l];
    const int C = L.c_in + L.c_out;
    const f32x4 *src = reinterpret_cast<const f32x4 *>(part_of(a.part, L) + static_cast<size_t>(bt) * C * (TT * KP));
    f32x4 x[KT], d[KT];   // all of a chunk's reads in flight at once
#pragma unroll
    for (int u = 0; u < KT; ++u) x[u] = d[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < L.c_in; ++c)
#pragma unroll
        for (int u = 0; u < KT; ++u) x[u] += src[static_cast<size_t>(c) * NQ + tid + 256 * u];
    for (int c = L.c_in; c < C; ++c)
#pragma unroll
        for (int u = 0; u < KT; ++u) d[u] += src[static_cast<size_t>(c) * NQ + tid + 256 * u];
#pragma unroll
    for (int u = 0; u < KT; ++u) {
        if constexpr (!kOwnX) xs[tid + 256 * u] = x[u];
        ds[tid + 256 * u] = d[u];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < KT * KT / NW; ++i) {
        const int blk = wave + NW * i;
        const int jo = blk / KT, ji = blk - jo * KT;
        f32x4 dv[MB], xv[MB];
#pragma unroll
        for (int m = 0; m < MB; ++m) {
            // own x': element (m KT + ji) 64 + lane = 256 u + 64 w + lane, u = (m KT + ji - w) / 4
            if constexpr (kOwnX) xv[m] = x[(m * KT + NW * i % KT) / NW];
            else xv[m] = xs[(m * KT + ji) * kWave + lane];
            dv[m] = ds[(m * KT + jo) * kWave + lane];
        }
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc = mfma16_f32(dv[m][r], xv[m][r], acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) gdst[blk * 256 + 64 * r] = acc[r];
    }
}

template <typename TOut>
__global__ __launch_bounds__(256) void k_project_reduce(ProjGroup grp, const float *gpart, const uint64_t *tile_bits,
                                                        int B, int tpe, int KT, int k_in, int k_out, int64_t g_ld) {
    // blockIdx.x: (layer, example); blockIdx.y: a 256-float block of the tile sums (block
    // (jo, ji) of G in the MFMA result layout: thread = 64 r + lane)
    const int l = blockIdx.x / B;
    const int b = blockIdx.x - l * B;
    const int KB = 256 * KT * KT;
    const int blk = blockIdx.y, jo = blk / KT, ji = blk - jo * KT;
    const int r = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int o = 16 * jo + 4 * (lane >> 4) + r, i = 16 * ji + (lane & 15);
    const float *p = gpart + static_cast<size_t>(l * B + b) * tpe * KB + blk * 256 + threadIdx.x;
    // tile_bits (or NULL): an empty tile's sum was never written; it counts as 0
    // (selected, so whatever the slot holds does not reach the sum)
    const uint64_t *tb = tile_bits ? tile_bits + static_cast<size_t>(b) * tpe : nullptr;
    auto kept = [&](int t, float v) { return tb == nullptr || load_uniform(tb + t) != 0 ? v : 0.f; };
    float s = 0.f;
    int t = 0;
    for (; t + 32 <= tpe; t += 32) {   // 32 loads in flight, summed in tile order
        float v[32];
#pragma unroll
        for (int u = 0; u < 32; ++u) v[u] = p[static_cast<size_t>(t + u) * KB];
#pragma unroll
        for (int u = 0; u < 32; ++u) s += kept(t + u, v[u]);
    }
    for (; t + 8 <= tpe; t += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = p[static_cast<size_t>(t + u) * KB];
#pragma unroll
        for (int u = 0; u < 8; ++u) s += kept(t + u, v[u]);
    }
    for (; t < tpe; ++t) s += kept(t, p[static_cast<size_t>(t) * KB]);
    if (o < k_out && i < k_in) {
        TOut *out = static_cast<TOut *>(grp.layer[l].g_out) + static_cast<int64_t>(b) * g_ld;
        store_out<TOut>(out + o * k_in + i, s);
    }
}

inline int kt_for(int k_in, int k_out) {
    const int kmax = k_in > k_out ? k_in : k_out;
    return kmax <= 16 ? 1 : kmax <= 32 ? 2 : kmax <= 64 ? 4 : 8;
}


struct Plan {
    size_t part_floats = 0, gpart_floats = 0;
    int slots = 0;
};

// Work items and workspace of a group; fills the per-layer fields of `a` if given.
Plan plan_group(const int *n_in, const int *n_out, int n_layers, int B, int T, int k_in, int k_out,
                ProjArgs *a) {
    const int KT = kt_for(k_in, k_out);
    const int ck = chunk_cols(KT);
    const int tpe = (T + TT - 1) / TT;
    Plan p;
    for (int l = 0; l < n_layers; ++l) {
        const int ci = (n_in[l] + ck - 1) / ck, co = (n_out[l] + ck - 1) / ck;
        if (a) {
            a->layer[l].n_in = n_in[l];
            a->layer[l].n_out = n_out[l];
            a->layer[l].c_in = static_cast<uint16_t>(ci);
            a->layer[l].c_out = static_cast<uint16_t>(co);
            a->layer[l].slot_begin = static_cast<uint16_t>(p.slots);
            a->layer[l].part_unit = static_cast<uint32_t>(p.part_floats / kPartUnit);
        }
        p.slots += ci + co;
        p.part_floats += static_cast<size_t>(ci + co) * B * tpe * TT * 16 * KT;
    }
    p.gpart_floats = static_cast<size_t>(n_layers) * B * tpe * (16 * KT) * (16 * KT);
    return p;
}

// Shared inputs: a layer whose x is the same tensor (same pointer and
// width) as an earlier layer's joins that layer's share set (up to
// kMaxShare; k <= 32 only), whose x items then project x once for every
// member.  Sets x_items, share_n, share and the work slots; returns the
// number of work slots and the largest share set.
int plan_shares(ProjArgs &a, int n_layers, int KT, int &smax) {
    smax = 1;
    for (int l = 0; l < n_layers; ++l) {
        ChunkLayer &L = a.layer[l];
        L.share_n = 0;
        int owner = -1;
        if (KT <= 2)
            for (int o = 0; o < l && owner < 0; ++o)
                if (a.layer[o].share_n > 0 && a.layer[o].share_n < kMaxShare && a.layer[o].x == L.x &&
                    a.layer[o].n_in == L.n_in)
                    owner = o;
        if (owner >= 0) {
            ChunkLayer &O = a.layer[owner];
            O.share[O.share_n++] = static_cast<uint8_t>(l);
            smax = O.share_n > smax ? O.share_n : smax;
            L.x_items = 0;
        } else {
            L.share_n = 1;
            L.share[0] = static_cast<uint8_t>(l);
            L.x_items = L.c_in;
        }
    }
    int slots = 0;
    for (int l = 0; l < n_layers; ++l) {
        a.layer[l].slot_begin = static_cast<uint16_t>(slots);
        slots += a.layer[l].x_items + a.layer[l].c_out;
    }
    return slots;
}

// Resident workgroups of a kernel on the current device (computed once per
// device and kernel).
template <void (*K)(ProjArgs), int kThreads = NT>
int resident_groups() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
    if (cache[dev] == 0) {
        int cus = 0, per_cu = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(K), kThreads, 0) !=
                hipSuccess ||
            per_cu <= 0)
            per_cu = 1;
        cache[dev] = cus * per_cu;
    }
    return cache[dev];
}

template <int KT, int S, typename TIn>
void launch_chunks_s(const ProjArgs &a, int max_items, hipStream_t s) {
    const int cap = resident_groups<k_project_chunks<KT, S, TIn>>();
    hipLaunchKernelGGL((k_project_chunks<KT, S, TIn>), dim3(max_items < cap ? max_items : cap), dim3(NT), 0, s, a);
}

template <int KT>
void launch_tiles(const ProjArgs &a, int max_items, hipStream_t s) {
    if constexpr (kTilePairs<KT>) {
        if (a.paired) {   // a unit is two items
            const int cap = resident_groups<k_project_tiles<KT, true>>();
            const int units = max_items / 2;
            hipLaunchKernelGGL((k_project_tiles<KT, true>), dim3(units < cap ? units : cap), dim3(NT), 0, s, a);
            return;
        }
    }
    const int cap = resident_groups<k_project_tiles<KT, false>>();
    hipLaunchKernelGGL((k_project_tiles<KT, false>), dim3(max_items < cap ? max_items : cap), dim3(NT), 0, s, a);
}

void launch_stream(const ProjArgs &a, int max_items, hipStream_t s) {
    const int cap = resident_groups<k_project_stream, kStreamNT>();
    const int units = a.paired ? max_items / 2 : max_items;   // the first unit of each workgroup is fixed
    hipLaunchKernelGGL(k_project_stream, dim3(units < cap ? units : cap), dim3(kStreamNT), 0, s, a);
}

// Tile groups sharing the projection slab (launch_tiles) for bf16 inputs at
// KT >= kTilesMinKT (k > 16) without shared inputs; the item-pipelined stream
// at k <= 16 without shared inputs; per-wave chunks otherwise.
constexpr int kTilesMinKT = 2;
template <int KT, typename TIn>
void launch_chunks(const ProjArgs &a, int max_items, int smax, hipStream_t s) {
    if constexpr (sizeof(TIn) == 2 && KT >= kTilesMinKT) {
        if (smax == 1) return launch_tiles<KT>(a, a.slots * ((a.B * a.tpe + NW - 1) / NW), s);
    }
    if constexpr (sizeof(TIn) == 2 && KT == 1) {
        if (smax == 1) return launch_stream(a, max_items, s);
    }
    if constexpr (KT <= 2) {
        if (smax == 3) return launch_chunks_s<KT, 3, TIn>(a, max_items, s);
        if (smax == 2) return launch_chunks_s<KT, 2, TIn>(a, max_items, s);
    }
    launch_chunks_s<KT, 1, TIn>(a, max_items, s);
}

static_assert(sizeof(ProjArgs) <= 3840, "kernel arguments must stay well under the 4 KB limit");

}  // namespace

size_t project_ws_bytes(const int *n_in, const int *n_out, int n_layers, int B, int T, int k_in,
                        int k_out) {
    if (n_layers <= 0 || B <= 0 || T <= 0) return 0;
    const Plan p = plan_group(n_in, n_out, n_layers, B, T, k_in, k_out, nullptr);
    const size_t tiles = static_cast<size_t>(B) * ((T + TT - 1) / TT);
    return align256(p.part_floats * sizeof(float)) + align256(p.gpart_floats * sizeof(float)) +
           align256((tiles + 2) * sizeof(int)) + 2 * align256(tiles * sizeof(uint64_t));
}

hipError_t launch_project(const ProjGroup &grp, bool bf16_in, int B, int T, const uint8_t *mask,
                          int k_in, int k_out, bool bf16_out, int64_t g_ld, void *ws, hipStream_t s) {
    if (B == 0 || T == 0 || grp.n_layers == 0) return hipSuccess;
    ProjArgs a;
    int n_in[kMaxGroup], n_out[kMaxGroup];
    for (int l = 0; l < grp.n_layers; ++l) {
        n_in[l] = grp.layer[l].n_in;
        n_out[l] = grp.layer[l].n_out;
        a.layer[l].x = grp.layer[l].x;
        a.layer[l].dy = grp.layer[l].dy;
        a.layer[l].p_in = grp.layer[l].p_in;
        a.layer[l].p_out = grp.layer[l].p_out;
    }
    const Plan p = plan_group(n_in, n_out, grp.n_layers, B, T, k_in, k_out, &a);
    // the compact layer table: partial offsets in 32-bit units, slot indices in 16 bits
    if (p.part_floats / kPartUnit > 0xffffffffull || p.slots > 0xffff) return hipErrorInvalidValue;
    const int KT = kt_for(k_in, k_out);
    a.n_layers = grp.n_layers;
    int smax = 1;
    a.slots = plan_shares(a, grp.n_layers, KT, smax);
    // Slots widest first (stable), so that the last items handed out are the
    // narrow ones and the tail after the last claim is short.
    a.ordered = a.slots <= kMaxSlots;
    // Paired: the stream kernel (bf16, k <= 16) or the tile-group kernel (bf16,
    // 16 < k <= 64), no shared inputs, one chunk per layer side, so a workgroup that
    // streams a tile's (or tile group's) x side and then its dy side forms the
    // tile sums itself and the tile-sum kernel is not launched; pairs widest first.
    a.paired = bf16_in && (KT == 1 || (KT >= kTilesMinKT && KT <= kMaxPairedKT)) && smax == 1 && a.ordered;
    for (int l = 0; l < grp.n_layers && a.paired; ++l) a.paired = a.layer[l].c_in == 1 && a.layer[l].c_out == 1;
    if (a.paired) {
        int order[kMaxGroup];
        for (int l = 0; l < grp.n_layers; ++l) order[l] = l;
        std::stable_sort(order, order + grp.n_layers, [&](int x, int y) {
            return a.layer[x].n_in + a.layer[x].n_out > a.layer[y].n_in + a.layer[y].n_out;
        });
        for (int r = 0; r < grp.n_layers; ++r)
            a.slot_order[r] = static_cast<uint16_t>(order[r] << 10 | a.layer[order[r]].slot_begin);
    } else if (a.ordered) {
        int width[kMaxSlots], layer_of[kMaxSlots];
        for (int l = 0; l < grp.n_layers; ++l) {
            const ChunkLayer &L = a.layer[l];
            for (int c = 0; c < L.x_items + L.c_out; ++c) {
                const int n = c < L.x_items ? L.n_in : L.n_out;
                const int col0 = (c < L.x_items ? c : c - L.x_items) * chunk_cols(KT);
                width[L.slot_begin + c] = min(chunk_cols(KT), n - col0);
                layer_of[L.slot_begin + c] = l;
            }
        }
        int n = 0;
        for (int w = chunk_cols(KT); w > 0; ) {   // descending distinct widths
            int next = 0;
            for (int sl = 0; sl < a.slots; ++sl) {
                if (width[sl] == w) a.slot_order[n++] = static_cast<uint16_t>(layer_of[sl] << 10 | sl);
                else if (width[sl] < w && width[sl] > next) next = width[sl];
            }
            w = next;
        }
    }
    a.mask = mask;
    char *w = static_cast<char *>(ws);
    a.part = reinterpret_cast<float *>(w);
    w += align256(p.part_floats * sizeof(float));
    a.gpart = reinterpret_cast<float *>(w);
    w += align256(p.gpart_floats * sizeof(float));
    a.B = B;
    a.T = T;
    a.tpe = (T + TT - 1) / TT;
    a.k_in = k_in;
    a.k_out = k_out;
    a.ck = chunk_cols(KT);
    const size_t ntiles = static_cast<size_t>(B) * a.tpe;
    int *list = reinterpret_cast<int *>(w);
    int *count = list + ntiles;
    uint64_t *bits = reinterpret_cast<uint64_t *>(w + align256((ntiles + 2) * sizeof(int)));
    uint64_t *tile_bits = reinterpret_cast<uint64_t *>(reinterpret_cast<char *>(bits) +
                                                       align256(ntiles * sizeof(uint64_t)));
    a.work = count + 1;
    a.tiles = mask ? list : nullptr;
    a.bits = mask ? bits : nullptr;
    a.tile_bits = mask ? tile_bits : nullptr;
    a.n_tiles = mask ? count : nullptr;
    hipLaunchKernelGGL(k_project_prep, dim3(1), dim3(1024), 0, s, mask, B, T, a.tpe, list, bits, tile_bits, count,
                       a.work);
    const int max_items = a.slots * B * a.tpe;
    switch (KT) {
        case 1: bf16_in ? launch_chunks<1, bf16_bits>(a, max_items, smax, s) : launch_chunks<1, float>(a, max_items, smax, s); break;
        case 2: bf16_in ? launch_chunks<2, bf16_bits>(a, max_items, smax, s) : launch_chunks<2, float>(a, max_items, smax, s); break;
        // k > 32, bf16: tile groups sharing each step's projection slab
        case 4: bf16_in ? launch_chunks<4, bf16_bits>(a, max_items, smax, s) : launch_chunks<4, float>(a, max_items, smax, s); break;
        default: bf16_in ? launch_chunks<8, bf16_bits>(a, max_items, smax, s) : launch_chunks<8, float>(a, max_items, smax, s); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int pairs = grp.n_layers * B * a.tpe * KT * KT;   // (tile, 16 x 16 block of G), one wave each
    const unsigned fgrid = static_cast<unsigned>((pairs + NW - 1) / NW);
    const unsigned tgrid = static_cast<unsigned>(grp.n_layers * B * a.tpe);   // one workgroup per tile
    switch (a.paired ? 0 : KT) {
        case 0: break;   // the stream kernel wrote the tile sums of the listed tiles
        case 1: hipLaunchKernelGGL((k_project_tile_finish<1>), dim3(fgrid), dim3(256), 0, s, a, pairs); break;
        case 2: hipLaunchKernelGGL((k_project_tile_finish_wg<2>), dim3(tgrid), dim3(256), 0, s, a); break;
        case 4: hipLaunchKernelGGL((k_project_tile_finish_wg<4>), dim3(tgrid), dim3(256), 0, s, a); break;
        default: hipLaunchKernelGGL((k_project_tile_finish_wg<8>), dim3(tgrid), dim3(256), 0, s, a); break;
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned grid = static_cast<unsigned>(grp.n_layers) * B;
    const unsigned blocks = static_cast<unsigned>(KT * KT);   // 16 x 16 blocks of G
    // paired with a mask: the sums of empty tiles were never written, the reduce skips them
    const uint64_t *skip = a.paired ? a.tile_bits : nullptr;
    if (bf16_out)
        hipLaunchKernelGGL((k_project_reduce<bf16_bits>), dim3(grid, blocks), dim3(256), 0, s, grp, a.gpart, skip, B,
                           a.tpe, KT, k_in, k_out, g_ld);
    else
        hipLaunchKernelGGL((k_project_reduce<float>), dim3(grid, blocks), dim3(256), 0, s, grp, a.gpart, skip, B,
                           a.tpe, KT, k_in, k_out, g_ld);
    return hipGetLastError();
}

}  // namespace logra
