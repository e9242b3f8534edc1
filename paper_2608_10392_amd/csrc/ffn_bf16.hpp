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
// mask lacks a block read a zero page instead, and each 16-row MFMA group
// skips the blocks none of its rows use. Pairs are sorted by mask key, so
// tiles hold similar masks.
//
// Engine shared by both kernels:
//  * 4 waves in a 2 x 2 arrangement; each wave owns TM/2 rows and half of
//    the tile's columns, in 16 x 16 MFMA groups (v_mfma_f32_16x16x32_bf16).
//  * The product is formed transposed, weights as the MFMA A operand and
//    token rows as B, so each lane accumulates consecutive output columns of
//    one row. The weight rows are placed in LDS so that 16-column groups 2J
//    and 2J + 1 interleave in blocks of 4: lane l then holds columns
//    32 J + 8 (l / 16) + 0..7 of row l % 16, written as one 16-byte store
//    (8 bf16 after GELU in the up kernel, 2 x 4 fp32 in the down kernel)
//    with no LDS staging.
//  * K is staged RB/2 deep: a stage holds RB-byte rows (64 or 128), and the
//    16-byte chunk c of row r sits at slot c ^ ((r >> 1) & (RB/16 - 1)).
//    Measured with the LDS bank-conflict counter on gfx950, both variants
//    make the fragment reads (16 rows x 4 chunks per instruction)
//    conflict-free at 4 cycles per 1 KB; the unswizzled layouts and a padded
//    144-byte stride run at half that rate or worse.
//  * Stages are filled by global_load_lds_dwordx4 (no register staging): one
//    instruction fills 1024/RB rows, each lane fetching the global chunk that
//    belongs in its swizzled slot. NST stages rotate; NST - 1 are in flight
//    while one is consumed. Waits are explicit vmcnt counts followed by a
//    bare s_barrier (a __syncthreads fence would drain every load).
//  * Tiles are sized so that two workgroups share a CU (OCC = 2): while one
//    waits on a barrier or runs its epilogue, the other keeps the matrix
//    cores busy.
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

// Staged-row geometry: RB bytes per row, K = RB/2 bf16 per stage.
template <int RB>
struct Stage {
    static constexpr int SK = RB / 2;
    static constexpr int CH = RB / 16;             // 16-byte chunks per row
    static constexpr int ROWS_PER_DMA = 1024 / RB;
    static constexpr int KSTEPS = SK / 32;          // MFMA K steps per stage
    __device__ static __forceinline__ int off(int r, int c) { return r * RB + ((c ^ ((r >> 1) & (CH - 1))) << 4); }
    // Row r and chunk c that lane `lane` fills when one DMA covers rows r0..
    __device__ static __forceinline__ void slot(int r0, int lane, int& r, int& c) {
        r = r0 + lane / CH;
        c = (lane % CH) ^ ((r >> 1) & (CH - 1));
    }
};

// Output column held by row m of 16-column MFMA group g (see the engine
// notes): groups 2J and 2J + 1 interleave in blocks of 4 columns.
__device__ __forceinline__ int group_col(int g, int m) {
    return 32 * (g >> 1) + 8 * (m >> 2) + (m & 3) + 4 * (g & 1);
}

// Dynamic LDS bytes of the two kernels: the stage ring, plus the row lists
// of the current and the next tile (up: tokens and pairs; down: block masks).
__host__ __device__ constexpr int up_lds_bytes(int TM, int M, int RB, int NST) { return NST * (TM + M) * RB + 16 * TM; }
__host__ __device__ constexpr int down_lds_bytes(int TM, int BN, int RB, int NST) { return NST * (TM + BN) * RB + 16 * TM; }

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

// Up-projection, persistent and pipelined across tiles.
//  * Ring of NST stages filled by buffer loads into LDS; a stage's
//    fragments are read into registers one stage ahead (two register sets),
//    so the matrix cores never wait on LDS latency and a slot is refilled as
//    soon as its fragments are in registers: NST - 1 stages stay in flight
//    while the next one is read.
//  * The ring runs on from one tile into the next: the next tile's first
//    stages are issued during the current tile's last iterations, and its
//    row lists (tokens, pairs) are copied to LDS at the current tile's first
//    iteration, so there is no cold prologue between tiles.
//  * Vector-memory operations complete in issue order for vmcnt: before a
//    stage is read, at most the loads issued after it (later stages, the
//    previous tile's epilogue stores, a row-list copy) may be outstanding.
//    Every epilogue store is issued (rows past the tile's count write the
//    sink row), so the count is exact.
template <int MW, int TM, int RB, int NST, int OCC>
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void up_kernel(UpParams p) {
    using S = Stage<RB>;
    static_assert(S::KSTEPS == 1, "one MFMA k step per stage");
    constexpr int M = MW * 32;
    constexpr int RG = TM / 32;                       // MFMA row groups per wave
    constexpr int LA = TM / S::ROWS_PER_DMA / 4;      // A copies per wave per stage
    constexpr int LB = M / S::ROWS_PER_DMA / 4;       // B copies per wave per stage
    constexpr int L = LA + LB;
    constexpr int NEPI = RG * (MW / 2);               // epilogue stores per wave
    constexpr int A_BYTES = TM * RB, STAGE = (TM + M) * RB, RING = NST * STAGE;
    static_assert(LA >= 1 && LB >= 1, "tile too small for one copy per wave");
    static_assert(TM * 4 <= 32 * 16, "a row list must fit one half-wave copy");
    static_assert(NST == 3, "the wait accounting is written for a 3-stage ring");
    constexpr int NFETCH = 1;                         // copies per wave for a tile's row lists
    static_assert(L + NEPI + NFETCH < 64, "vmcnt range");
    extern __shared__ __attribute__((aligned(16))) char lds_up[];
    // rows[par][0] tokens, rows[par][1] pairs of the tile with parity par
    int* rows = reinterpret_cast<int*>(lds_up + RING);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int n_tiles = ld_uniform(p.totals + 1);
    const int nk = p.d / S::SK;     // stages per tile: even, and >= NST + 1 (d >= 128)
    int tile = xcd_tile(0);
    if (tile >= n_tiles) return;

    // Fragment addresses inside a stage: lane (lr, lg) reads row base + lr,
    // chunk lg; 16-row steps keep the swizzle, so row groups are constant
    // offsets from these.
    const int lr = lane & 15, lg = lane >> 4;
    const uint32_t fa = S::off(wm * (TM / 2) + lr, lg);
    const uint32_t fb = A_BYTES + S::off(wn * (M / 2) + lr, lg);
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
        voffB[j] = (uint32_t)group_col(r >> 4, r & 15) * row_bytes + ch * 16;
    }
    const char* srcA[LA];   // token rows of the tile being issued
    size_t wslab = 0;       // byte offset of that tile's weight slab

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
        wslab = ((size_t)e * p.H + (size_t)c * M) * row_bytes;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            int r, ch;
            S::slot((wave * LA + j) * S::ROWS_PER_DMA, lane, r, ch);
            const int tok = (r < nrows) ? rows[par * 2 * TM + r] : 0;
            srcA[j] = reinterpret_cast<const char*>(p.X) + (size_t)tok * row_bytes + ch * 16;
        }
    };
    // Ring slots of the next stage to issue and of the next stage to read,
    // and the k offset (bytes) of the next stage to issue.
    int slot_w = 0, slot_r = 0;
    uint32_t k_w = 0;
    int issued = 0;
    // The copies of one stage (q < LA: token rows, the rest weight rows),
    // issued one at a time between MFMAs (see step).
    auto issue_one = [&](int q) {
        char* base = lds_up + slot_w * STAGE;
        if (q < LA) dma16(srcA[q] + k_w, base + (wave * LA + q) * 1024);
        else dma16(wup + (wslab + k_w) + voffB[q - LA], base + A_BYTES + (wave * LB + q - LA) * 1024);
    };
    auto issue_end = [&]() {
        slot_w = (slot_w == NST - 1) ? 0 : slot_w + 1;
        k_w += S::SK * 2;
        ++issued;
    };
    auto issue = [&]() {
#pragma unroll
        for (int q = 0; q < L; ++q) issue_one(q);
        issue_end();
    };
    // Fragments are kept as raw 32-bit words (bf16 vectors in loop-carried
    // registers make the compiler split them into halves).
    u32x4 a0[RG], b0[MW], a1[RG], b1[MW];
    auto load_frags = [&](u32x4 (&A)[RG], u32x4 (&Bw)[MW]) {
        const char* st = lds_up + slot_r * STAGE;
#pragma unroll
        for (int j = 0; j < MW; ++j) Bw[j] = ld16(st + fb + j * 16 * RB);
#pragma unroll
        for (int i = 0; i < RG; ++i) A[i] = ld16(st + fa + i * 16 * RB);
        slot_r = (slot_r == NST - 1) ? 0 : slot_r + 1;
    };
    f32x4 acc[RG][MW];

    int par = 0;
    int info = ld_uniform(p.tile_info + tile);
    fetch_rows(tile, 0);
    wait_vmcnt<0>();
    __syncthreads();
    sources(0, info);
    for (int ks = 0; ks < NST; ++ks) issue();
    wait_vmcnt<(NST - 1) * L>();
    __builtin_amdgcn_s_barrier();
    load_frags(a0, b0);
    wait_lgkmcnt0();
    bool after_epi = false;
    for (int round = 0;; ++round) {
        const int next = xcd_tile(round + 1);
        const bool has_next = next < n_tiles;
        const int next_info = has_next ? ld_uniform(p.tile_info + next) : 0;
#pragma unroll
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        // Fragments of tile stage s are in (A, Bw): wait for stage s + 1,
        // refill the slot freed by stage s with the stage NST ahead (of this
        // tile, of the next tile, or - past the last tile - a harmless
        // re-read of this tile's first stages into the free slot, which
        // keeps every iteration's copy count the same), read stage s + 1
        // into (A2, B2), then run stage s.
        // FIRST marks s = 0 and 1, where the previous tile's epilogue stores
        // (issued after stages 0..NST-1 of this tile) and the row-list copy
        // (issued at s = 0, before stage NST) sit behind the awaited stage.
        auto step = [&](auto first, int s, u32x4 (&A)[RG], u32x4 (&Bw)[MW], u32x4 (&A2)[RG],
                        u32x4 (&B2)[MW]) {
            if constexpr (decltype(first)::value) {
                const int n_after = L + (after_epi ? NEPI : 0) + ((s == 1 && has_next) ? NFETCH : 0);
                wait_vm_after<L, NEPI, NFETCH>(n_after);
            } else {
                wait_vmcnt<L>();
            }
            __builtin_amdgcn_s_barrier();
            if (s == 0 && has_next) fetch_rows(next, par ^ 1);
            if (s + NST == nk) {
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
            load_frags(A2, B2);
            // MFMAs by row group, with the stage's copies spread between them.
#pragma unroll
            for (int i = 0; i < RG; ++i) {
#pragma unroll
                for (int j = 0; j < MW; ++j) acc[i][j] = mfma16x16x32(as_bf16x8(Bw[j]), as_bf16x8(A[i]), acc[i][j]);
#pragma unroll
                for (int q = 0; q < L; ++q)
                    if (q * RG / L == i) issue_one(q);
                __builtin_amdgcn_sched_barrier(0);
            }
            issue_end();
            // The fragments just read must be in registers before the next
            // barrier lets another wave refill their slot.
            wait_lgkmcnt0();
        };
        step(std::true_type{}, 0, a0, b0, a1, b1);
        step(std::true_type{}, 1, a1, b1, a0, b0);
        for (int s = 2; s < nk; s += 2) {
            step(std::false_type{}, s, a0, b0, a1, b1);
            step(std::false_type{}, s + 1, a1, b1, a0, b0);
        }
        // GELU, round to bf16; lane stores 8 consecutive columns of its row.
        const int sl = info & 0xffff, nrows = info >> 16;
        const int c = sl - (sl / p.B) * p.B;
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int r = wm * (TM / 2) + i * 16 + (lane & 15);
            u16* dst = (r < nrows) ? p.Hbuf + (size_t)rows[(par * 2 + 1) * TM + r] * p.H + (size_t)c * M : p.Hsink;
            dst += wn * (M / 2) + 8 * (lane >> 4);
#pragma unroll
            for (int J = 0; J < MW / 2; ++J) {
                const f32x4 lo = acc[i][2 * J], hi = acc[i][2 * J + 1];
                u32x4 v;
                v[0] = pack_bf16x2(gelu_as7126(lo[0]), gelu_as7126(lo[1]));
                v[1] = pack_bf16x2(gelu_as7126(lo[2]), gelu_as7126(lo[3]));
                v[2] = pack_bf16x2(gelu_as7126(hi[0]), gelu_as7126(hi[1]));
                v[3] = pack_bf16x2(gelu_as7126(hi[2]), gelu_as7126(hi[3]));
                st16(dst + 32 * J, v);
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

// Down-projection on the same engine as the up kernel (ring of buffer
// loads, fragments read one stage ahead, pipelined across tiles). A tile is
// TM consecutive pairs of one expert x BN output columns; its stages walk
// the blocks of the tile's mask union, M/32 stages per block. A row whose
// mask lacks the stage's block reads zeros (an out-of-range offset), and a
// 16-row MFMA group whose rows all lack it skips its MFMAs. Tiles with fewer
// than NST + 1 stages are padded with empty stages (no MFMAs), so the ring
// never runs more than one tile ahead.
template <int NW, int TM, int RB, int NST, int OCC>
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void down_kernel(DownParams p) {
    using S = Stage<RB>;
    static_assert(S::KSTEPS == 1, "one MFMA k step per stage");
    constexpr int BN = NW * 32;
    constexpr int RG = TM / 32;                       // MFMA row groups per wave
    constexpr int G = TM / 16;                        // 16-row groups per tile
    constexpr int LA = TM / S::ROWS_PER_DMA / 4;
    constexpr int LB = BN / S::ROWS_PER_DMA / 4;
    constexpr int L = LA + LB;
    constexpr int NEPI = RG * NW;                     // epilogue stores per wave
    constexpr int A_BYTES = TM * RB, STAGE = (TM + BN) * RB, RING = NST * STAGE;
    static_assert(LA >= 1 && LB >= 1, "tile too small for one copy per wave");
    constexpr int NFETCH = TM * 8 / 256;              // 4-byte copies per wave for a tile's row masks
    static_assert(NST == 3, "the wait accounting is written for a 3-stage ring");
    static_assert(L + NEPI + NFETCH < 64, "vmcnt range");
    extern __shared__ __attribute__((aligned(16))) char lds_dn[];
    uint64_t* rmask = reinterpret_cast<uint64_t*>(lds_dn + RING);   // [2][TM]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int n_tiles = ld_uniform(p.totals + 2);
    const int kcpb = p.M / S::SK;   // stages per block (even: M is a multiple of 64)
    int tile = xcd_tile(0);
    if (tile >= n_tiles) return;

    const int lr = lane & 15, lg = lane >> 4;
    const uint32_t fa = S::off(wm * (TM / 2) + lr, lg);
    const uint32_t fb = A_BYTES + S::off(wn * (BN / 2) + lr, lg);
    const uint32_t hrow = (uint32_t)p.H * 2;
    const char* const wdn = reinterpret_cast<const char*>(p.Wdown);
    uint32_t voffB[LB], vA[LA];
    int rA[LA];
#pragma unroll
    for (int j = 0; j < LB; ++j) {
        int r, ch;
        S::slot((wave * LB + j) * S::ROWS_PER_DMA, lane, r, ch);
        voffB[j] = (uint32_t)group_col(r >> 4, r & 15) * hrow + ch * 16;
    }
#pragma unroll
    for (int j = 0; j < LA; ++j) {
        int ch;
        S::slot((wave * LA + j) * S::ROWS_PER_DMA, lane, rA[j], ch);
        vA[j] = (uint32_t)rA[j] * hrow + ch * 16;
    }

    // Uniform description of a tile.
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
        const uint64_t* ms = p.rt_masks + (size_t)rt * (G + 1);
        D.all = ld_uniform64(ms + G);
#pragma unroll
        for (int i = 0; i < RG; ++i) D.gm[i] = ld_uniform64(ms + wm * RG + i);
        D.nreal = __popcll(D.all) * kcpb;
        D.nst = max(D.nreal, NST + 1);
        return D;
    };
    // A tile's row masks (TM u64) are copied to LDS by every wave, in
    // 4-byte pieces (a tile's first pair can be any index).
    auto fetch_masks = [&](Desc D, int par) {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(p.pair_mask + D.p0);
#pragma unroll
        for (int q = 0; q < NFETCH; ++q) dma4(src + q * 64 + lane, rmask + par * TM + q * 32);
    };

    // Issue side: the tile whose stages are being copied.
    const char* hbase = reinterpret_cast<const char*>(p.Hbuf);
    uint64_t mrow[LA];
    size_t wbase = 0;
    uint64_t rem_w = 0;
    int cb_w = 0, kc_w = 0, st_w = 0, nreal_w = 0;
    auto issue_tile = [&](Desc D, int par) {
        hbase = reinterpret_cast<const char*>(p.Hbuf + (size_t)D.p0 * p.H);
#pragma unroll
        for (int j = 0; j < LA; ++j) mrow[j] = (rA[j] < D.nrows) ? rmask[par * TM + rA[j]] : 0ull;
        wbase = ((size_t)D.e * p.d + (size_t)D.ct * BN) * hrow;
        rem_w = D.all;
        cb_w = rem_w ? __builtin_ctzll(rem_w) : 0;
        kc_w = 0;
        st_w = 0;
        nreal_w = D.nreal;
    };
    int slot_w = 0, slot_r = 0, issued = 0;
    // The copies of one stage: copy q < LA fills A rows, the rest B rows.
    // They are issued one at a time between MFMAs (see step), so that a
    // copy held up at the texture unit never leaves the matrix cores idle.
    char* cp_base = lds_dn;
    uint32_t cp_soff = 0;
    bool cp_real = false;
    auto issue_begin = [&]() {
        cp_base = lds_dn + slot_w * STAGE;
        cp_real = st_w < nreal_w;
        cp_soff = (uint32_t)(cb_w * p.M + kc_w * S::SK) * 2;
    };
    auto issue_one = [&](int q) {
        if (q < LA)
            dma16((cp_real && ((mrow[q] >> cb_w) & 1ull)) ? hbase + (vA[q] + cp_soff) : reinterpret_cast<const char*>(p.zero16),
                  cp_base + (wave * LA + q) * 1024);
        else
            dma16(wdn + (wbase + cp_soff) + voffB[q - LA], cp_base + A_BYTES + (wave * LB + q - LA) * 1024);
    };
    auto issue_end = [&]() {
        slot_w = (slot_w == NST - 1) ? 0 : slot_w + 1;
        ++issued;
        ++st_w;
        if (++kc_w == kcpb) {
            kc_w = 0;
            rem_w &= rem_w - 1;
            cb_w = rem_w ? __builtin_ctzll(rem_w) : 0;
        }
    };
    auto issue = [&]() {
        issue_begin();
#pragma unroll
        for (int q = 0; q < L; ++q) issue_one(q);
        issue_end();
    };
    u32x4 a0[RG], b0[NW], a1[RG], b1[NW];
    auto load_frags = [&](u32x4 (&A)[RG], u32x4 (&Bw)[NW]) {
        const char* st = lds_dn + slot_r * STAGE;
#pragma unroll
        for (int j = 0; j < NW; ++j) Bw[j] = ld16(st + fb + j * 16 * RB);
#pragma unroll
        for (int i = 0; i < RG; ++i) A[i] = ld16(st + fa + i * 16 * RB);
        slot_r = (slot_r == NST - 1) ? 0 : slot_r + 1;
    };
    f32x4 acc[RG][NW];

    int par = 0;
    Desc cur = describe(tile);
    fetch_masks(cur, 0);
    wait_vmcnt<0>();
    __syncthreads();
    issue_tile(cur, 0);
    for (int q = 0; q < NST; ++q) issue();
    wait_vmcnt<(NST - 1) * L>();
    __builtin_amdgcn_s_barrier();
    load_frags(a0, b0);
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
            for (int j = 0; j < NW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        // Read side: block and stage of the stage in registers.
        uint64_t rem_r = cur.all;
        int cb_r = rem_r ? __builtin_ctzll(rem_r) : 0, kc_r = 0;
        const int nst = cur.nst;
        // Same step as the up kernel; the MFMAs of a row group run only if
        // one of its rows uses the stage's block.
        auto step = [&](auto first, int s, u32x4 (&A)[RG], u32x4 (&Bw)[NW], u32x4 (&A2)[RG],
                        u32x4 (&B2)[NW]) {
            if constexpr (decltype(first)::value) {
                const int n_after = L + (after_epi ? NEPI : 0) + ((s == 1 && has_next) ? NFETCH : 0);
                wait_vm_after<L, NEPI, NFETCH>(n_after);
            } else {
                wait_vmcnt<L>();
            }
            __builtin_amdgcn_s_barrier();
            if (s == 0 && has_next) fetch_masks(nxt, par ^ 1);
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
            issue_begin();
            load_frags(A2, B2);
            const bool real = s < cur.nreal;
#pragma unroll
            for (int i = 0; i < RG; ++i) {
                if (real && ((cur.gm[i] >> cb_r) & 1ull)) {
#pragma unroll
                    for (int j = 0; j < NW; ++j)
                        acc[i][j] = mfma16x16x32(as_bf16x8(Bw[j]), as_bf16x8(A[i]), acc[i][j]);
                }
#pragma unroll
                for (int q = 0; q < L; ++q)
                    if (q * RG / L == i) issue_one(q);
                __builtin_amdgcn_sched_barrier(0);
            }
            issue_end();
            if (++kc_r == kcpb) {
                kc_r = 0;
                rem_r &= rem_r - 1;
                cb_r = rem_r ? __builtin_ctzll(rem_r) : 0;
            }
            // The fragments just read must be in registers before the next
            // barrier lets another wave refill their slot.
            wait_lgkmcnt0();
        };
        step(std::true_type{}, 0, a0, b0, a1, b1);
        step(std::true_type{}, 1, a1, b1, a0, b0);
        for (int s = 2; s < nst; s += 2) {
            step(std::false_type{}, s, a0, b0, a1, b1);
            step(std::false_type{}, s + 1, a1, b1, a0, b0);
        }
        // fp32 per-expert rows; lane stores 8 consecutive columns of its row.
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int r = wm * (TM / 2) + i * 16 + lr;
            float* dst = (r < cur.nrows) ? p.part + (size_t)(cur.p0 + r) * p.d + (size_t)cur.ct * BN : p.part_sink;
            dst += wn * (BN / 2) + 8 * lg;
#pragma unroll
            for (int J = 0; J < NW / 2; ++J) {
                st16(dst + 32 * J, __builtin_bit_cast(u32x4, acc[i][2 * J]));
                st16(dst + 32 * J + 4, __builtin_bit_cast(u32x4, acc[i][2 * J + 1]));
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
