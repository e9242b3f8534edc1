// Block-sparse expert FFN on the bf16 matrix cores (Eq. block-expert-output).
//
// Up-projection + GELU, one tile = TM rows of one (expert e, block c) slab:
//   Hbuf[pair, c M .. c M + M) = GELU(X[token(pair)] K_e[:, block c])
// Rows come from the slab's compacted pair list, so no inactive (pair, block)
// is computed. The tile spans the whole block width M, so each gathered token
// row is read once per slab.
//
// Down-projection, one tile = TM consecutive pairs of one expert segment x
// BN output columns:
//   part[pair, n] = sum over blocks c of the pair's mask of
//                   Hbuf[pair, block c] . V_e[block c, n]        (fp32)
// The contraction runs over the union of the tile's block masks; rows whose
// mask lacks a block read a zero page instead, and each 32-row MFMA group
// skips the blocks none of its rows use. Pairs are sorted by mask key, so
// tiles hold similar masks.
//
// Engine shared by both kernels:
//  * One workgroup of 4 waves per CU, 2 x 2: each wave owns TM/2 rows and
//    half of the tile's columns, in 32 x 32 MFMA groups
//    (v_mfma_f32_32x32x16_bf16: one wave per SIMD keeps the matrix core
//    busier with these than with 16 x 16 groups, and the 32-cycle issue
//    shadow hides the copies, LDS reads and bookkeeping).
//  * The product is formed transposed, weights as the MFMA A operand and
//    token rows as B, so each lane accumulates output columns of one row.
//    Weight rows are placed in LDS so that lane l of a 32-column group holds
//    columns 16 (l / 32) + 0..15 (see wcol): 16 consecutive values of one
//    row, written as 16-byte stores with no LDS staging.
//  * K is staged 64 deep: a stage holds one 128-byte line per row, so every
//    L2 request of the copies is a whole line (half-line requests ran at
//    half the bytes per clock on gfx950). The 16-byte chunk c of row r sits
//    at slot c ^ ((r >> 1) & 7), which keeps the fragment reads (32 rows x 2
//    chunks per instruction) free of LDS bank conflicts.
//  * Stages are filled by global_load_lds_dwordx4 (no register staging): one
//    instruction fills 8 rows, each lane fetching the global chunk that
//    belongs in its swizzled slot. NST stages rotate; NST - 1 are in flight
//    while one is consumed. Waits are explicit vmcnt counts followed by a
//    bare s_barrier (a __syncthreads fence would drain every load).
//  * Persistent over a device-built tile table, with consecutive tiles mapped
//    to workgroups of the same XCD (dispatch is round-robin over 8 XCDs), so
//    co-running tiles share weight slabs in that XCD's L2.
#pragma once
#include <type_traits>
#include "common.hpp"

namespace unifmoe {

constexpr int kFfnThreads = 256;
constexpr int kXcds = 8;

struct UpParams {
    int d, M, B, H;
    const u16* X;
    const u16* Wup;
    u16* Hbuf;
    u16* Hsink;              // one H row that absorbs the stores of a tile's unused rows
    const int* slab_rows;    // pair of each slab row
    const int* slab_tok;
    const int* tile_info;    // slab | rows << 16
    const int* tile_rows;    // first entry of the tile's rows in slab_rows / slab_tok
    const int* totals;
};

struct DownParams {
    int d, M, B, H, ncol;        // ncol: column tiles per row tile
    const u16* Hbuf;
    const u16* zero16;           // 16 zero bytes: the source of rows that lack a block
    const u16* Wdown;
    float* part;
    float* part_sink;            // one d row that absorbs the stores of unused tile rows
    const int4* rt_info;         // per row tile: first pair, rows, expert
    const uint64_t* rt_masks;    // per row tile: block-mask union of each 16-row group, then of the tile
    const uint64_t* pair_mask;   // readable for a whole tile past the last pair
    const int* tiles;            // per down tile: row tile << 8 | column tile
    const int* totals;           // [2]: down tiles
};

// Staged-row geometry: one 128-byte line (64 bf16 of k) per row and stage.
struct Stage {
    static constexpr int RB = 128;
    static constexpr int SK = 64;                  // k per stage
    static constexpr int CH = 8;                   // 16-byte chunks per row
    static constexpr int ROWS_PER_DMA = 8;         // rows filled by one 1-KB copy
    static constexpr int KSTEPS = 4;               // 16-deep MFMA steps per stage
    __device__ static __forceinline__ uint32_t off(int r, int c) { return r * RB + ((c ^ ((r >> 1) & 7)) << 4); }
    // Row r and chunk c that lane `lane` fills when one copy covers rows r0..
    __device__ static __forceinline__ void slot(int r0, int lane, int& r, int& c) {
        r = r0 + lane / CH;
        c = (lane % CH) ^ ((r >> 1) & 7);
    }
};

// Output column (within its 32-column group) of the weight row staged at
// position r of the group. The MFMA gives lane l the D rows
// 8 j + 4 (l / 32) + i in accumulator element 4 j + i; with this order those
// rows are the columns 16 (l / 32) + 4 j + i.
__device__ __forceinline__ int wcol(int r) { return 16 * ((r >> 2) & 1) + 4 * (r >> 3) + (r & 3); }

// Dynamic LDS bytes of the two kernels: the stage ring, plus the row lists
// of the current and the next tile (up: tokens and pairs; down: block masks).
__host__ __device__ constexpr int up_lds_bytes(int TM, int M, int NST) { return NST * (TM + M) * Stage::RB + 16 * TM; }
__host__ __device__ constexpr int down_lds_bytes(int TM, int BN, int NST) { return NST * (TM + BN) * Stage::RB + 16 * TM; }

// Tile handled by this workgroup in persistent round `round`: a contiguous
// range of tiles per XCD. gridDim.x is a multiple of kXcds.
__device__ __forceinline__ int xcd_tile(int round) {
    const int per = gridDim.x / kXcds;
    return round * gridDim.x + (blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
}

// Wait until at most n vector-memory operations of this wave are pending,
// for the few counts the GEMM pipelines use (anything else waits for all).
template <int L, int E, int F>
__device__ __forceinline__ void wait_vm_after(int n) {
    if (n == L) wait_vmcnt<L>();
    else if (n == L + F) wait_vmcnt<L + F>();
    else if (n == L + E) wait_vmcnt<L + E>();
    else if (n == L + E + F) wait_vmcnt<L + E + F>();
    else if (n == E) wait_vmcnt<E>();
    else if (n == E + F) wait_vmcnt<E + F>();
    else if (n == F) wait_vmcnt<F>();
    else wait_vmcnt<0>();
}

// Wait before step s of a tile reads stage s + 1. Issued after that stage:
// the later stages still in flight (NST - 2 of them), and in the first
// NST - 1 steps also the previous tile's epilogue stores (issued after stage
// NST - 1) and, from step 1 on, the next tile's row-list copy (issued at
// step 0, before stage NST).
template <int NST, int L, int NEPI, int NFETCH>
__device__ __forceinline__ void wait_stage(bool first, int s, bool after_epi, bool has_next) {
    if (first && s <= NST - 2) {
        const int n = (NST - 2) * L + (after_epi ? NEPI : 0) + ((s >= 1 && has_next) ? NFETCH : 0);
        wait_vm_after<(NST - 2) * L, NEPI, NFETCH>(n);
    } else {
        wait_vmcnt<(NST - 2) * L>();
    }
}

// Up-projection, persistent and pipelined across tiles.
//  * Ring of NST stages filled by copies into LDS; a stage's fragments are
//    read into registers one stage ahead (two register sets), so the matrix
//    cores never wait on LDS latency and a slot is refilled as soon as its
//    fragments are in registers: NST - 1 stages stay in flight while the
//    next one is read.
//  * The ring runs on from one tile into the next: the next tile's first
//    stages are issued during the current tile's last iterations, and its
//    row lists (tokens, pairs) are copied to LDS at the current tile's first
//    iteration, so there is no cold prologue between tiles.
//  * Vector-memory operations complete in issue order for vmcnt: before a
//    stage is read, at most the loads issued after it (later stages, the
//    previous tile's epilogue stores, a row-list copy) may be outstanding.
//    Every epilogue store is issued (rows past the tile's count write the
//    sink row), so the count is exact.
//  * A tile has nk = d / 64 stages; tiles shorter than NST + 1 stages are
//    padded with stages that re-read k = 0.. and run no MFMAs.
template <int MG, int TM, int NST>
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void up_kernel(UpParams p) {
    using S = Stage;
    constexpr int RB = S::RB, KS = S::KSTEPS;
    constexpr int M = MG * 64;                        // MG 32-column groups per wave
    constexpr int RG = TM / 64;                       // 32-row groups per wave
    constexpr int LA = TM / S::ROWS_PER_DMA / 4;      // token-row copies per wave per stage
    constexpr int LB = M / S::ROWS_PER_DMA / 4;       // weight-row copies per wave per stage
    constexpr int L = LA + LB;
    constexpr int NEPI = RG * MG * 2;                 // epilogue stores per wave
    constexpr int A_BYTES = TM * RB, STAGE = (TM + M) * RB, RING = NST * STAGE;
    constexpr int NU = KS * RG;                       // MFMA units per stage
    static_assert(LA >= 1 && LB >= 1, "tile too small for one copy per wave");
    static_assert(TM * 4 <= 32 * 16, "a row list must fit one half-wave copy");
    static_assert(NST >= 3 && NST <= 5, "ring depth");
    constexpr int NFETCH = 1;                         // copies per wave for a tile's row lists
    static_assert((NST - 2) * L + NEPI + NFETCH < 64, "vmcnt range");
    extern __shared__ __attribute__((aligned(16))) char lds_up[];
    // rows[par][0] tokens, rows[par][1] pairs of the tile with parity par
    int* rows = reinterpret_cast<int*>(lds_up + RING);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int n_tiles = ld_uniform(p.totals + 1);
    const int nk = p.d / S::SK;                       // real stages per tile (even)
    const int nst = (max(nk, NST + 1) + 1) & ~1;      // stages per tile, padding included (even)
    int tile = xcd_tile(0);
    if (tile >= n_tiles) return;

    // Fragment addresses inside a stage: lane (lr, lh) reads row base + lr,
    // chunk 2 k + lh of k step k; 32-row steps keep the swizzle, so row
    // groups are constant offsets from these.
    const int lr = lane & 31, lh = lane >> 5;
    uint32_t fx[KS], fw[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) {
        fx[k] = S::off(wm * (TM / 2) + lr, 2 * k + lh);
        fw[k] = A_BYTES + S::off(wn * (M / 2) + lr, 2 * k + lh);
    }
    // Copy sources: per-lane addresses fixed for a tile, plus the k position
    // (and, for weights, the slab) as a uniform byte offset. Token rows past
    // the tile's count read token 0; their results go to the sink row.
    const uint32_t row_bytes = (uint32_t)p.d * 2;
    const char* const wup = reinterpret_cast<const char*>(p.Wup);
    uint32_t voffB[LB];
#pragma unroll
    for (int j = 0; j < LB; ++j) {
        int r, ch;
        S::slot((wave * LB + j) * S::ROWS_PER_DMA, lane, r, ch);
        voffB[j] = (uint32_t)(32 * (r >> 5) + wcol(r & 31)) * row_bytes + ch * 16;
    }
    const char* srcA[LA];   // token rows of the tile being issued
    const char* wslab = wup;

    // A tile's token and pair lists (TM ints each) are copied by waves 0/2
    // and 1/3 (both copies of a list land on the same bytes), so that every
    // wave issues the same number of vector-memory operations.
    auto fetch_rows = [&](int t, int par) {
        if (lane < TM / 4) {
            const int which = wave & 1;
            const int* src = (which == 0 ? p.slab_tok : p.slab_rows) + ld_uniform(p.tile_rows + t) + lane * 4;
            dma16(src, rows + (par * 2 + which) * TM);
        }
    };
    auto sources = [&](int par, int inf) {
        const int sl = inf & 0xffff, nrows = inf >> 16;
        const int e = sl / p.B, c = sl - e * p.B;
        wslab = wup + ((size_t)e * p.H + (size_t)c * M) * row_bytes;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            int r, ch;
            S::slot((wave * LA + j) * S::ROWS_PER_DMA, lane, r, ch);
            const int tok = (r < nrows) ? rows[par * 2 * TM + r] : 0;
            srcA[j] = reinterpret_cast<const char*>(p.X) + (size_t)tok * row_bytes + ch * 16;
        }
    };
    // Ring slot (byte offset) of the next stage to issue and of the next
    // stage to read, and the k offset (bytes) of the next stage to issue.
    uint32_t slot_w = 0, slot_r = 0;
    uint32_t k_w = 0;
    auto issue_one = [&](int q) {
        char* base = lds_up + slot_w;
        if (q < LA) dma16(srcA[q] + k_w, base + (wave * LA + q) * 1024);
        else dma16(wslab + k_w + voffB[q - LA], base + A_BYTES + (wave * LB + q - LA) * 1024);
    };
    auto issue_end = [&]() {
        slot_w = (slot_w == (NST - 1) * STAGE) ? 0u : slot_w + STAGE;
        k_w += RB;
        if (k_w == row_bytes) k_w = 0;    // padding stages re-read the row start
    };
    auto issue = [&]() {
#pragma unroll
        for (int q = 0; q < L; ++q) issue_one(q);
        issue_end();
    };
    // Fragments are kept as raw 32-bit words (bf16 vectors in loop-carried
    // registers make the compiler split them into halves).
    u32x4 x0[KS][RG], w0[KS][MG], x1[KS][RG], w1[KS][MG];
    // Fragment read r of a stage: k step r / (MG + RG), then its MG weight
    // and RG token fragments.
    constexpr int NR = KS * (MG + RG);
    auto read_one = [&](const char* st, int r, u32x4 (&X)[KS][RG], u32x4 (&W)[KS][MG]) {
        const int k = r / (MG + RG), t = r % (MG + RG);
        if (t < MG) W[k][t] = ld16(st + fw[k] + t * 32 * RB);
        else X[k][t - MG] = ld16(st + fx[k] + (t - MG) * 32 * RB);
    };
    auto next_slot_r = [&]() { slot_r = (slot_r == (NST - 1) * STAGE) ? 0u : slot_r + STAGE; };
    auto load_frags = [&](u32x4 (&X)[KS][RG], u32x4 (&W)[KS][MG]) {
#pragma unroll
        for (int r = 0; r < NR; ++r) read_one(lds_up + slot_r, r, X, W);
        next_slot_r();
    };
    f32x16 acc[RG][MG];

    int par = 0;
    int info = ld_uniform(p.tile_info + tile);
    fetch_rows(tile, 0);
    wait_vmcnt<0>();
    __syncthreads();
    sources(0, info);
    for (int ks = 0; ks < NST; ++ks) issue();
    wait_vmcnt<(NST - 1) * L>();
    __builtin_amdgcn_s_barrier();
    load_frags(x0, w0);
    wait_lgkmcnt0();
    bool after_epi = false;
    for (int round = 0;; ++round) {
        const int next = xcd_tile(round + 1);
        const bool has_next = next < n_tiles;
        const int next_info = has_next ? ld_uniform(p.tile_info + next) : 0;
#pragma unroll
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int j = 0; j < MG; ++j) acc[i][j] = f32x16{};
        // Fragments of tile stage s are in (X, W): wait for stage s + 1,
        // refill the slot freed by stage s with the stage NST ahead (of this
        // tile, of the next tile, or - past the last tile - a harmless
        // re-read of this tile's first stages into the free slot, which
        // keeps every iteration's copy count the same), read stage s + 1
        // into (X2, W2), then run stage s.
        // FIRST marks s = 0 and 1, where the previous tile's epilogue stores
        // (issued after stages 0..NST-1 of this tile) and the row-list copy
        // (issued at s = 0, before stage NST) sit behind the awaited stage.
        auto step = [&](auto first, int s, u32x4 (&X)[KS][RG], u32x4 (&W)[KS][MG], u32x4 (&X2)[KS][RG],
                        u32x4 (&W2)[KS][MG]) {
            wait_stage<NST, L, NEPI, NFETCH>(decltype(first)::value, s, after_epi, has_next);
            __builtin_amdgcn_s_barrier();
            if constexpr (decltype(first)::value) {
                if (s == 0 && has_next) fetch_rows(next, par ^ 1);
            }
            if (s + NST == nst) {
                // From here on the stages issued belong to the next tile.
                // Its row lists were copied at s == 0, before stage NST,
                // which has been waited for when s >= NST - 1.
                if (has_next) {
                    if (s < NST - 1) {
                        wait_vmcnt<0>();
                        __builtin_amdgcn_s_barrier();
                    }
                    sources(par ^ 1, next_info);
                }
                k_w = 0;
            }
            const char* st2 = lds_up + slot_r;
            next_slot_r();
            const bool real = s < nk;
            // MFMAs by (k step, row group), with the reads of stage s + 1's
            // fragments and the copies of stage s + NST spread between them
            // (no reads after the last group, so they have landed by the
            // step's end).
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int k = u / RG, i = u % RG;
                if (real) {
#pragma unroll
                    for (int j = 0; j < MG; ++j)
                        acc[i][j] = mfma32x32x16(as_bf16x8(W[k][j]), as_bf16x8(X[k][i]), acc[i][j]);
                }
#pragma unroll
                for (int r = 0; r < NR; ++r)
                    if (r * (NU - 1) / NR == u) read_one(st2, r, X2, W2);
#pragma unroll
                for (int q = 0; q < L; ++q)
                    if (q * NU / L == u) issue_one(q);
                __builtin_amdgcn_sched_barrier(0);
            }
            issue_end();
            // The fragments just read must be in registers before the next
            // barrier lets another wave refill their slot.
            wait_lgkmcnt0();
        };
        // Steps 0 .. NST - 2 carry the first-steps wait accounting; nst is
        // even and at least NST + 1.
        step(std::true_type{}, 0, x0, w0, x1, w1);
        step(std::true_type{}, 1, x1, w1, x0, w0);
        int s = 2;
        if constexpr (NST >= 4) {
            step(std::true_type{}, 2, x0, w0, x1, w1);
            step(std::true_type{}, 3, x1, w1, x0, w0);
            s = 4;
        }
        for (; s < nst; s += 2) {
            step(std::false_type{}, s, x0, w0, x1, w1);
            step(std::false_type{}, s + 1, x1, w1, x0, w0);
        }
        // GELU, round to bf16; lane stores 16 consecutive columns of its row
        // per 32-column group.
        const int sl = info & 0xffff, nrows = info >> 16;
        const int c = sl - (sl / p.B) * p.B;
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int r = wm * (TM / 2) + i * 32 + lr;
            u16* dst = (r < nrows) ? p.Hbuf + (size_t)rows[(par * 2 + 1) * TM + r] * p.H + (size_t)c * M : p.Hsink;
            dst += wn * (M / 2) + 16 * lh;
#pragma unroll
            for (int j = 0; j < MG; ++j) {
                const f32x16 v = acc[i][j];
                u32x4 lo, hi;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    lo[t] = pack_bf16x2(gelu_as7126(v[2 * t]), gelu_as7126(v[2 * t + 1]));
                    hi[t] = pack_bf16x2(gelu_as7126(v[8 + 2 * t]), gelu_as7126(v[9 + 2 * t]));
                }
                st16(dst + 32 * j, lo);
                st16(dst + 32 * j + 8, hi);
            }
        }
        if (!has_next) break;
        info = next_info;
        par ^= 1;
        after_epi = true;
    }
    // The re-reads issued past the last tile land in LDS: let them finish
    // before the workgroup's LDS is released.
    wait_vmcnt<0>();
}

// Down-projection on the same engine as the up kernel (ring of copies,
// fragments read one stage ahead, pipelined across tiles). A tile is TM
// consecutive pairs of one expert x BN output columns; its stages walk the
// blocks of the tile's mask union, M/64 stages per block. A row whose mask
// lacks the stage's block reads the zero page, and a 32-row MFMA group whose
// rows all lack it skips its MFMAs. Tiles are padded to an even number of at
// least NST + 1 stages with empty stages (no MFMAs), so the ring never runs
// more than one tile ahead.
template <int NG, int TM, int NST>
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void down_kernel(DownParams p) {
    using S = Stage;
    constexpr int RB = S::RB, KS = S::KSTEPS;
    constexpr int BN = NG * 64;                       // NG 32-column groups per wave
    constexpr int RG = TM / 64;                       // 32-row groups per wave
    constexpr int G16 = TM / 16;                      // 16-row mask groups per tile
    constexpr int LA = TM / S::ROWS_PER_DMA / 4;
    constexpr int LB = BN / S::ROWS_PER_DMA / 4;
    constexpr int L = LA + LB;
    constexpr int NEPI = RG * NG * 4;                 // epilogue stores per wave
    constexpr int A_BYTES = TM * RB, STAGE = (TM + BN) * RB, RING = NST * STAGE;
    constexpr int NU = KS * RG;
    static_assert(LA >= 1 && LB >= 1, "tile too small for one copy per wave");
    constexpr int NFETCH = TM * 8 / 256;              // 4-byte copies per wave for a tile's row masks
    static_assert(NST >= 3 && NST <= 5, "ring depth");
    static_assert((NST - 2) * L + NEPI + NFETCH < 64, "vmcnt range");
    extern __shared__ __attribute__((aligned(16))) char lds_dn[];
    uint64_t* rmask = reinterpret_cast<uint64_t*>(lds_dn + RING);   // [2][TM]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int n_tiles = ld_uniform(p.totals + 2);
    const int kcpb = p.M / S::SK;   // stages per block
    int tile = xcd_tile(0);
    if (tile >= n_tiles) return;

    const int lr = lane & 31, lh = lane >> 5;
    uint32_t fx[KS], fw[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) {
        fx[k] = S::off(wm * (TM / 2) + lr, 2 * k + lh);
        fw[k] = A_BYTES + S::off(wn * (BN / 2) + lr, 2 * k + lh);
    }
    const uint32_t hrow = (uint32_t)p.H * 2;
    const uint32_t blk_bytes = (uint32_t)p.M * 2;
    const char* const wdn = reinterpret_cast<const char*>(p.Wdown);
    const char* const zero = reinterpret_cast<const char*>(p.zero16);
    uint32_t voffB[LB], vA[LA];
    int rA[LA];
#pragma unroll
    for (int j = 0; j < LB; ++j) {
        int r, ch;
        S::slot((wave * LB + j) * S::ROWS_PER_DMA, lane, r, ch);
        voffB[j] = (uint32_t)(32 * (r >> 5) + wcol(r & 31)) * hrow + ch * 16;
    }
#pragma unroll
    for (int j = 0; j < LA; ++j) {
        int ch;
        S::slot((wave * LA + j) * S::ROWS_PER_DMA, lane, rA[j], ch);
        vA[j] = (uint32_t)rA[j] * hrow + ch * 16;
    }

    // Uniform description of a tile; gm[i]: block mask of this wave's
    // 32-row group i.
    struct Desc {
        int p0, nrows, e, ct, nst, nreal;
        uint64_t all, gm[RG];
    };
    auto describe = [&](int t) {
        Desc D;
        const int rc = ld_uniform(p.tiles + t);
        const int rt = rc >> 8;
        D.ct = rc & 255;
        const int* inf = reinterpret_cast<const int*>(p.rt_info + rt);
        D.p0 = ld_uniform(inf);
        D.nrows = ld_uniform(inf + 1);
        D.e = ld_uniform(inf + 2);
        const uint64_t* ms = p.rt_masks + (size_t)rt * (G16 + 1);
        D.all = ld_uniform64(ms + G16);
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int g = 2 * (wm * RG + i);
            D.gm[i] = ld_uniform64(ms + g) | ld_uniform64(ms + g + 1);
        }
        D.nreal = __popcll(D.all) * kcpb;
        D.nst = (max(D.nreal, NST + 1) + 1) & ~1;
        return D;
    };
    // A tile's row masks (TM u64) are copied to LDS by every wave, in
    // 4-byte pieces (a tile's first pair can be any index).
    auto fetch_masks = [&](Desc D, int par) {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(p.pair_mask + D.p0);
#pragma unroll
        for (int q = 0; q < NFETCH; ++q) dma4(src + q * 64 + lane, rmask + par * TM + q * 32);
    };

    // Issue side. Per block, each H-row copy either walks its row (one
    // stage of k per stage) or re-reads the zero page (stride 0); the weight
    // copies walk the expert's rows from a uniform base. Past the last block
    // of the union (padding stages) the H copies read the zero page and the
    // weight copies re-read block 0 (in range, never used).
    const char* hbase = nullptr;
    const char* wtile = wdn;
    uint64_t mrow[LA];
    const char* pa[LA];
    uint32_t sa[LA];
    const char* pb = wdn;
    uint64_t rem_w = 0;
    int kc_w = 0;
    auto set_block_w = [&]() {
        const uint64_t low = rem_w & (0ull - rem_w);
        const int cb = rem_w ? __builtin_ctzll(rem_w) : 0;
        pb = wtile + (size_t)cb * blk_bytes;
#pragma unroll
        for (int q = 0; q < LA; ++q) {
            const bool on = (mrow[q] & low) != 0;
            pa[q] = on ? hbase + (vA[q] + (uint32_t)cb * blk_bytes) : zero;
            sa[q] = on ? (uint32_t)RB : 0u;
        }
    };
    auto issue_tile = [&](Desc D, int par) {
        hbase = reinterpret_cast<const char*>(p.Hbuf + (size_t)D.p0 * p.H);
#pragma unroll
        for (int j = 0; j < LA; ++j) mrow[j] = (rA[j] < D.nrows) ? rmask[par * TM + rA[j]] : 0ull;
        // Settle the mask reads here, so that no later use waits on them
        // behind the fragment reads of a step.
        wait_lgkmcnt0();
        wtile = wdn + ((size_t)D.e * p.d + (size_t)D.ct * BN) * hrow;
        rem_w = D.all;
        kc_w = 0;
        set_block_w();
    };
    uint32_t slot_w = 0, slot_r = 0;
    // The copies of one stage: copy q < LA fills H rows, the rest weight
    // rows. They are issued one at a time between MFMAs (see step).
    auto issue_one = [&](int q) {
        char* base = lds_dn + slot_w;
        if (q < LA) dma16(pa[q], base + (wave * LA + q) * 1024);
        else dma16(pb + voffB[q - LA], base + A_BYTES + (wave * LB + q - LA) * 1024);
    };
    auto issue_end = [&]() {
        slot_w = (slot_w == (NST - 1) * STAGE) ? 0u : slot_w + STAGE;
#pragma unroll
        for (int q = 0; q < LA; ++q) pa[q] += sa[q];
        pb += RB;
        if (++kc_w == kcpb) {
            kc_w = 0;
            rem_w &= rem_w - 1;
            set_block_w();
        }
    };
    auto issue = [&]() {
#pragma unroll
        for (int q = 0; q < L; ++q) issue_one(q);
        issue_end();
    };
    u32x4 x0[KS][RG], w0[KS][NG], x1[KS][RG], w1[KS][NG];
    constexpr int NR = KS * (NG + RG);
    auto read_one = [&](const char* st, int r, u32x4 (&X)[KS][RG], u32x4 (&W)[KS][NG]) {
        const int k = r / (NG + RG), t = r % (NG + RG);
        if (t < NG) W[k][t] = ld16(st + fw[k] + t * 32 * RB);
        else X[k][t - NG] = ld16(st + fx[k] + (t - NG) * 32 * RB);
    };
    auto next_slot_r = [&]() { slot_r = (slot_r == (NST - 1) * STAGE) ? 0u : slot_r + STAGE; };
    auto load_frags = [&](u32x4 (&X)[KS][RG], u32x4 (&W)[KS][NG]) {
#pragma unroll
        for (int r = 0; r < NR; ++r) read_one(lds_dn + slot_r, r, X, W);
        next_slot_r();
    };
    f32x16 acc[RG][NG];

    int par = 0;
    Desc cur = describe(tile);
    fetch_masks(cur, 0);
    wait_vmcnt<0>();
    __syncthreads();
    issue_tile(cur, 0);
    for (int q = 0; q < NST; ++q) issue();
    wait_vmcnt<(NST - 1) * L>();
    __builtin_amdgcn_s_barrier();
    load_frags(x0, w0);
    wait_lgkmcnt0();
    bool after_epi = false;
    for (int round = 0;; ++round) {
        const int next = xcd_tile(round + 1);
        const bool has_next = next < n_tiles;
        Desc nxt;
        if (has_next) nxt = describe(next);
#pragma unroll
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int j = 0; j < NG; ++j) acc[i][j] = f32x16{};
        // Read side: which of this wave's row groups use the block of the
        // stage in registers (bit i: group i), and the stage within it.
        // After the last block the set is empty (padding stages).
        uint64_t rem_r = cur.all;
        int kc_r = 0;
        auto groups = [&]() {
            const uint64_t low = rem_r & (0ull - rem_r);
            uint32_t g = 0;
#pragma unroll
            for (int i = 0; i < RG; ++i) g |= ((cur.gm[i] & low) != 0 ? 1u : 0u) << i;
            return g;
        };
        uint32_t gset = groups();
        const int nst = cur.nst;
        auto step = [&](auto first, int s, u32x4 (&X)[KS][RG], u32x4 (&W)[KS][NG], u32x4 (&X2)[KS][RG],
                        u32x4 (&W2)[KS][NG]) {
            wait_stage<NST, L, NEPI, NFETCH>(decltype(first)::value, s, after_epi, has_next);
            __builtin_amdgcn_s_barrier();
            if constexpr (decltype(first)::value) {
                if (s == 0 && has_next) fetch_masks(nxt, par ^ 1);
            }
            if (s + NST == nst) {
                // From here on the stages issued belong to the next tile (or,
                // past the last tile, re-read this tile's first stages into
                // the free slot). The next tile's row masks were copied at
                // s == 0, before stage NST, waited for when s >= NST - 1.
                if (has_next && s < NST - 1) {
                    wait_vmcnt<0>();
                    __builtin_amdgcn_s_barrier();
                }
                Desc D = cur;
                if (has_next) D = nxt;
                issue_tile(D, has_next ? par ^ 1 : par);
            }
            const char* st2 = lds_dn + slot_r;
            next_slot_r();
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int k = u / RG, i = u % RG;
                if (gset & (1u << i)) {
#pragma unroll
                    for (int j = 0; j < NG; ++j)
                        acc[i][j] = mfma32x32x16(as_bf16x8(W[k][j]), as_bf16x8(X[k][i]), acc[i][j]);
                }
#pragma unroll
                for (int r = 0; r < NR; ++r)
                    if (r * (NU - 1) / NR == u) read_one(st2, r, X2, W2);
#pragma unroll
                for (int q = 0; q < L; ++q)
                    if (q * NU / L == u) issue_one(q);
                __builtin_amdgcn_sched_barrier(0);
            }
            issue_end();
            if (++kc_r == kcpb) {
                kc_r = 0;
                rem_r &= rem_r - 1;
                gset = groups();
            }
            // The fragments just read must be in registers before the next
            // barrier lets another wave refill their slot.
            wait_lgkmcnt0();
        };
        // Steps 0 .. NST - 2 carry the first-steps wait accounting; nst is
        // even and at least NST + 1.
        step(std::true_type{}, 0, x0, w0, x1, w1);
        step(std::true_type{}, 1, x1, w1, x0, w0);
        int s = 2;
        if constexpr (NST >= 4) {
            step(std::true_type{}, 2, x0, w0, x1, w1);
            step(std::true_type{}, 3, x1, w1, x0, w0);
            s = 4;
        }
        for (; s < nst; s += 2) {
            step(std::false_type{}, s, x0, w0, x1, w1);
            step(std::false_type{}, s + 1, x1, w1, x0, w0);
        }
        // fp32 per-expert rows; lane stores 16 consecutive columns of its row
        // per 32-column group.
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int r = wm * (TM / 2) + i * 32 + lr;
            float* dst = (r < cur.nrows) ? p.part + (size_t)(cur.p0 + r) * p.d + (size_t)cur.ct * BN : p.part_sink;
            dst += wn * (BN / 2) + 16 * lh;
#pragma unroll
            for (int j = 0; j < NG; ++j) {
                const f32x16 v = acc[i][j];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    u32x4 w;
                    w[0] = __float_as_uint(v[4 * t]);
                    w[1] = __float_as_uint(v[4 * t + 1]);
                    w[2] = __float_as_uint(v[4 * t + 2]);
                    w[3] = __float_as_uint(v[4 * t + 3]);
                    st16(dst + 32 * j + 4 * t, w);
                }
            }
        }
        if (!has_next) break;
        cur = nxt;
        par ^= 1;
        after_epi = true;
    }
    // The re-reads issued past the last tile land in LDS: let them finish
    // before the workgroup's LDS is released.
    wait_vmcnt<0>();
}

}  // namespace unifmoe
