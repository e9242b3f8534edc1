// Block-sparse expert FFN on the matrix cores (Eq. block-expert-output).
//
// Up-projection + GELU (bf16 products), one tile = TM rows of one (expert e,
// block c) slab:
//   Hbuf[pair, c M .. c M + M) = fp16(GELU(X[token(pair)] K_e[:, block c]))
// Rows come from the slab's compacted pair list, so no inactive (pair, block)
// is computed. The tile spans the whole block width M, so each gathered token
// row is read once per slab.
//
// Down-projection (fp16 products: the activations H and a fp16 copy of the
// bf16 values V, which fp16 holds exactly down to 2^-17 in magnitude), one
// tile = TM consecutive pairs of one expert segment x BN output columns:
//   part[pair, n] = sum over blocks c of the pair's mask of
//                   Hbuf[pair, block c] . V_e[block c, n]        (fp32)
// H is kept in fp16 rather than bf16 because its rounding enters every
// output through a sum over all active channels: with bf16 (relative step
// 2^-8) it alone takes a sixth of the bf16 output bound on these layers,
// with fp16 (2^-11) an eighth of that.
// The contraction runs over the union of the tile's block masks; rows whose
// mask lacks a block read a zero page instead, and each 32-row MFMA group
// skips the blocks none of its rows use. Pairs are sorted by mask key, so
// tiles hold similar masks.
//
// Engine shared by both kernels:
//  * One workgroup of 8 waves per CU (two per SIMD), 4 x 2: each wave owns
//    64 of the tile's 256 rows and half of its columns, in 32 x 32 MFMA
//    groups (v_mfma_f32_32x32x16_bf16). The 256-row tile is what the copy
//    path of a CU can feed: the bytes staged per MFMA flop fall by a third
//    against 128-row tiles.
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
//    belongs in its swizzled slot. Two stage slots alternate. Fragments are
//    read from LDS one 16-deep k step ahead into two register sets; before
//    the last k step of stage s the waves wait for stage s + 1 and meet at
//    a barrier, after which every wave holds all of stage s in registers, so
//    its slot is refilled with stage s + 2 while stage s + 1 is consumed.
//    Waits are explicit vmcnt counts followed by a bare s_barrier (a
//    __syncthreads fence would drain every load).
//  * Persistent over a device-built tile table. Each XCD (dispatch is
//    round-robin over 8 XCDs) owns one contiguous eighth of the table, and
//    its workgroups take the next tile from a per-XCD counter as they free
//    up, so consecutive tiles run side by side on one XCD and share its L2
//    (weight slabs, and the H rows a row tile's column tiles all read).
//    Which workgroup computes a tile does not change its result.
#pragma once
#include <type_traits>
#include "common.hpp"

namespace unifmoe {

constexpr int kFfnThreads = 512;
constexpr int kFfnWaves = 8;
constexpr int kFfnTM = 256;   // rows per tile (4 waves x 2 groups of 32)

// What the up kernel does with its fp32 tile a (rows x the block's M
// channels) of one (expert, block) slab:
//   kEpiGelu      H = fp16(GELU(a))                       (forward)
//   kEpiGeluBias  H = fp16(GELU(a + b1))                   (block forward)
//   kEpiPre       H = fp16(a)                              (backward, a = x K^T)
//   kEpiDa        with g = dy V (rows read from dY, weights V^T), w the
//                 pair weight and a = H: dcp = partial sums of GELU(a) . g
//                 (the pair's d loss / d w = dy . E restricted to the
//                 block), G = bf16(w g GELU'(a)) = d loss / d(x K^T) and
//                 H = bf16(w GELU(a)), in place          (backward)
constexpr int kEpiGelu = 0, kEpiGeluBias = 1, kEpiPre = 2, kEpiDa = 3;

struct UpParams {
    int d, M, B, H;
    const u16* X;            // token rows (dY for kEpiDa)
    const u16* Wup;          // [K+1, H, d] (V^T for kEpiDa)
    u16* Hbuf;
    u16* Hsink;              // one H row that absorbs the stores of a tile's unused rows
    const int* slab_rows;    // pair of each slab row
    const int* slab_tok;
    const int* tile_info;    // slab | rows << 16
    const int* tile_rows;    // first entry of the tile's rows in slab_rows / slab_tok
    const int* totals;
    int* queue;              // 8 per-XCD tile counters, zero at launch
    const float* b_up;       // [K+1, H] fp32 biases added before the GELU (kEpiGeluBias only)
    u16* Gbuf;               // kEpiDa: layout of Hbuf (its sink row included)
    const float* pw;         // kEpiDa: weight of each pair
    float* dcp;              // kEpiDa: [pairs + 1, B, 2] partial sums (block, column half)
    int sink_row;            // kEpiDa: the pair slot whose rows of Hbuf, Gbuf and dcp absorb a
                             // tile's unused rows (Hsink's row)
};

struct DownParams {
    int d, M, B, H, ncol;        // ncol: column tiles per row tile
    const u16* Hbuf;             // fp16 (F16 kernels) or bf16
    const u16* zero16;           // 16 zero bytes: the source of rows that lack a block
    const u16* Wdown;            // values V in Hbuf's format, layout of the layer's W_down
    float* part;                 // per-pair output rows, fp32
    float* part_sink;            // one d row that absorbs the stores of unused tile rows
    const int4* rt_info;         // per row tile: first pair, rows, expert
    const uint64_t* rt_masks;    // per row tile: block-mask union of each 32-row group, then of the tile
    const uint64_t* pair_mask;   // readable for a whole tile past the last pair
    const int* slices;           // [kXcds + 1]: the tiles (row tile x column tile x part) of each XCD's queue
    int* queue;                  // 8 per-XCD tile counters, zero at launch
    int nsplit;                  // parts each tile's block union is split into by block index mod nsplit (1: none)
    size_t split_stride;         // floats between the parts' row buffers in part
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

// Dynamic LDS bytes of the two kernels: two stage slots, plus the row lists
// of the current and the next tile (up: tokens and pairs; down: block masks).
// The last 16 bytes pass tile indices between waves.
__host__ __device__ constexpr int up_lds_bytes(int M, int TM) { return 2 * (TM + M) * Stage::RB + 16 * TM + 16; }
__host__ __device__ constexpr int down_lds_bytes(int TM, int BN) { return 2 * (TM + BN) * Stage::RB + 16 * TM + 16; }

// Per-XCD tile queue: XCD x (= blockIdx.x % 8) owns tiles [lo, hi) of the
// table and hands them out in order through counter queue[x]. Indices past
// hi mean "no tile". gridDim.x is a multiple of kXcds.
struct TileQueue {
    int* ctr;
    int lo, hi;
    __device__ TileQueue(int* queue, int n_tiles) {
        const int x = blockIdx.x % kXcds;
        ctr = queue + x;
        lo = (int)((int64_t)x * n_tiles / kXcds);
        hi = (int)((int64_t)(x + 1) * n_tiles / kXcds);
    }
    // Slices given by a table: XCD x owns [slices[x], slices[x + 1]).
    __device__ TileQueue(int* queue, const int* slices) {
        const int x = blockIdx.x % kXcds;
        ctr = queue + x;
        lo = ld_uniform(slices + x);
        hi = ld_uniform(slices + x + 1);
    }
    // One lane only (a vector atomic with return); the result is an offset
    // from lo.
    __device__ int take(int n) const { return atomicAdd(ctr, n); }
};

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

// Wait at the barrier of stage s of a tile, for stage s + 1. Only stage
// s + 1 is in flight then, plus what was issued after it: at s = 0 the
// previous tile's epilogue stores, at s = 1 the next tile's row-list copy.
template <int NEPI, int NFETCH>
__device__ __forceinline__ void wait_stage(int s, bool after_epi, bool has_next) {
    const int n = (s == 0 && after_epi) ? NEPI : ((s == 1 && has_next) ? NFETCH : 0);
    wait_vm_after<0, NEPI, NFETCH>(n);
}

// Up-projection, persistent and pipelined across tiles.
//  * The copies run on from one tile into the next: the next tile's first
//    two stages are issued during the current tile's last two stages, and
//    its row lists (tokens, pairs) are copied to LDS during stage 0, so
//    there is no cold prologue between tiles.
//  * Vector-memory operations complete in issue order for vmcnt; every
//    epilogue store is issued (rows past the tile's count write the sink
//    row), so the counts are exact.
//  * A tile has nk = d / 64 stages; tiles shorter than 4 stages are padded
//    with stages that re-read k = 0.. and run no MFMAs (the row-list copy of
//    stage 0 is waited for at the barrier of stage 2). PAD: whether d < 256
//    (else no stage is padding and the MFMAs need no per-stage test).
template <int MG, bool PAD, int TM, int EPI = kEpiGelu>
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void up_kernel(UpParams p) {
    using S = Stage;
    constexpr int RB = S::RB, KS = S::KSTEPS, NWV = kFfnWaves;
    constexpr int M = MG * 64;                        // MG 32-column groups per wave
    constexpr int RG = TM / 128;                      // 32-row groups per wave (4 row waves)
    static_assert(TM == 256 || TM == 384, "tile heights with whole row-list copies");
    constexpr int LA = TM / S::ROWS_PER_DMA / NWV;    // token-row copies per wave per stage
    constexpr int LB = M / S::ROWS_PER_DMA / NWV;     // weight-row copies per wave per stage
    constexpr int L = LA + LB;
    // Epilogue stores per wave: H (two per 32-column group), and G for
    // kEpiDa, which also stores its partial sums and first loads H, whose
    // waits (placed by the compiler) drain the copies in flight; so NEPI is
    // a lower bound of what follows the copies there.
    constexpr int NEPI = RG * MG * (EPI == kEpiDa ? 4 : 2);
    constexpr int A_BYTES = TM * RB, STAGE = (TM + M) * RB, RING = 2 * STAGE;
    // 4-byte copies per wave for a tile's row lists (2 TM ints): one of 64
    // ints per wave, and for TM = 384 one more of 32.
    constexpr int NFETCH = (2 * TM > NWV * 64) ? 2 : 1;
    constexpr int NR = RG + MG;                       // fragment reads per k step
    static_assert(LA >= 1 && LB >= 1, "tile too small for one copy per wave");
    static_assert(2 * TM == NWV * 64 || 2 * TM == NWV * 96, "row lists: one or one and a half copies per wave");
    static_assert(NEPI + NFETCH + L < 64, "vmcnt range");
    extern __shared__ __attribute__((aligned(16))) char lds_up[];
    // rows[par][0] tokens, rows[par][1] pairs of the tile with parity par
    int* rows = reinterpret_cast<int*>(lds_up + RING);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int n_tiles = ld_uniform(p.totals + 1);
    const int nk = p.d / S::SK;                       // real stages per tile
    const int nst = max(nk, 4);                       // stages per tile, padding included
    const TileQueue tq(p.queue, n_tiles);
    // ctl[0], ctl[1]: the first two tiles; ctl[2]: the tile after next,
    // taken at stage 0 of each tile, written at stage 1, read after stage 2.
    int* ctl = reinterpret_cast<int*>(lds_up + RING + 16 * TM);
    if (tid == 0) {
        const int t = tq.take(2);
        ctl[0] = t;
        ctl[1] = t + 1;
    }
    __syncthreads();
    int tile = tq.lo + __builtin_amdgcn_readfirstlane(ctl[0]);
    int next = tq.lo + __builtin_amdgcn_readfirstlane(ctl[1]);
    if (tile >= tq.hi) return;
    int taken = 0;

    // Fragment addresses inside a stage: lane (lr, lh) reads row base + lr,
    // chunk 2 k + lh of k step k; 32-row steps keep the swizzle, so row
    // groups are constant offsets from these.
    const int lr = lane & 31, lh = lane >> 5;
    uint32_t fx[KS], fw[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) {
        fx[k] = S::off(wm * (TM / 4) + lr, 2 * k + lh);
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

    // A tile's token and pair lists (TM ints each, stored back to back):
    // wave w copies ints 64 w .. 64 w + 63 of the two lists, and for TM = 384
    // also ints 512 + 32 w .. (pairs 128 + 32 w ..), so that every wave issues
    // the same number of operations.
    auto fetch_rows = [&](int first, int par) {
        int* dst = rows + par * 2 * TM;
        const int i0 = wave * 64;   // the list boundary TM is a multiple of 64
        dma4((i0 < TM ? p.slab_tok + first + i0 : p.slab_rows + first + (i0 - TM)) + lane, dst + i0);
        if constexpr (NFETCH == 2) {
            const int i1 = NWV * 64 + wave * 32;
            if (lane < 32) dma4(p.slab_rows + first + (i1 - TM) + lane, dst + i1);
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
    // k offset (bytes) of the next stage to issue.
    uint32_t k_w = 0;
    auto issue_one = [&](uint32_t slot, int q) {
        char* base = lds_up + slot;
        if (q < LA) dma16(srcA[q] + k_w, base + (wave * LA + q) * 1024);
        else dma16(wslab + k_w + voffB[q - LA], base + A_BYTES + (wave * LB + q - LA) * 1024);
    };
    auto issue_end = [&]() {
        k_w += RB;
        if (k_w == row_bytes) k_w = 0;    // padding stages re-read the row start
    };
    // Fragments are kept as raw 32-bit words (bf16 vectors in loop-carried
    // registers make the compiler split them into halves).
    u32x4 fxa[RG], fwa[MG], fxb[RG], fwb[MG];
    auto read_one = [&](uint32_t slot, int k, int r, u32x4 (&X)[RG], u32x4 (&W)[MG]) {
        const char* st = lds_up + slot;
        if (r < MG) W[r] = ld16(st + fw[k] + r * 32 * RB);
        else X[r - MG] = ld16(st + fx[k] + (r - MG) * 32 * RB);
    };
    f32x16 acc[RG][MG];

    int par = 0;
    int info = ld_uniform(p.tile_info + tile);
    fetch_rows(ld_uniform(p.tile_rows + tile), 0);
    wait_vmcnt<0>();
    __syncthreads();
    sources(0, info);
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
        for (int q = 0; q < L; ++q) issue_one(st * STAGE, q);
        issue_end();
    }
    wait_vmcnt<L>();
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int r = 0; r < NR; ++r) read_one(0, 0, r, fxa, fwa);
    uint32_t slot = 0;          // slot of the stage being computed
    bool after_epi = false;
    for (;;) {
        const bool has_next = next < tq.hi;
        const int next_info = has_next ? ld_uniform(p.tile_info + next) : 0;
        const int next_rows = has_next ? ld_uniform(p.tile_rows + next) : 0;
        // No scalar load may be in flight in the stage loop: the compiler
        // can then wait for the fragment reads of one k step only (lgkmcnt
        // also counts scalar loads, which complete out of order).
        wait_lgkmcnt0();
#pragma unroll
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int j = 0; j < MG; ++j) acc[i][j] = f32x16{};
        for (int s = 0; s < nst; ++s) {
            const bool real = !PAD || s < nk;
            const uint32_t other = slot ^ STAGE;
            // k step k: reads of the next k step into (X2, W2) first (a
            // whole k step of MFMAs covers their latency), then the MFMAs on
            // (X, W) by row group; the last k step also issues stage s + 2
            // into this stage's slot, between the row groups.
            auto kstep = [&](int k, u32x4 (&X)[RG], u32x4 (&W)[MG], u32x4 (&X2)[RG], u32x4 (&W2)[MG]) {
                const uint32_t rslot = (k == KS - 1) ? other : slot;
                const int rk = (k == KS - 1) ? 0 : k + 1;
#pragma unroll
                for (int r = 0; r < NR; ++r) read_one(rslot, rk, r, X2, W2);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < RG; ++i) {
                    if (real) {
#pragma unroll
                        for (int j = 0; j < MG; ++j)
                            acc[i][j] = mfma32x32x16(as_bf16x8(W[j]), as_bf16x8(X[i]), acc[i][j]);
                    }
                    if (k == KS - 1) {
#pragma unroll
                        for (int q = 0; q < L; ++q)
                            if (q * RG / L == i) issue_one(slot, q);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            };
            kstep(0, fxa, fwa, fxb, fwb);
            kstep(1, fxb, fwb, fxa, fwa);
            kstep(2, fxa, fwa, fxb, fwb);
            // Stage s is in registers once the k step 3 reads land; stage
            // s + 1 once this wave's copies of it have, and for all waves
            // after the barrier.
            wait_lgkmcnt0();
            wait_stage<NEPI, NFETCH>(s, after_epi, has_next);
            __builtin_amdgcn_s_barrier();
            // The atomic is issued before stage s + 2's copies, so the wait
            // of stage 1 (for stage 2) covers it.
            if (s == 0 && has_next && tid == 0) taken = tq.take(1);
            if (s == 1 && has_next && tid == 0) ctl[2] = taken;
            if (s + 2 == nst) {
                // The stages issued from here on belong to the next tile, or,
                // past the last tile, re-read this tile's first ones.
                sources(has_next ? par ^ 1 : par, has_next ? next_info : info);
                k_w = 0;
            }
            kstep(3, fxb, fwb, fxa, fwa);
            issue_end();
            if (s == 0 && has_next) fetch_rows(next_rows, par ^ 1);
            slot = other;
        }
        // GELU, round to fp16; lane stores 16 consecutive columns of its row
        // per 32-column group.
        const int sl = info & 0xffff, nrows = info >> 16;
        const int c = sl - (sl / p.B) * p.B;
        if constexpr (EPI == kEpiPre) {
#pragma unroll
            for (int i = 0; i < RG; ++i) {
                const int r = wm * (TM / 4) + i * 32 + lr;
                const bool live = r < nrows;
                const int pr = live ? rows[(par * 2 + 1) * TM + r] : 0;
                const size_t off = (live ? (size_t)pr * p.H + (size_t)c * M : 0) + wn * (M / 2) + 16 * lh;
                u16* ha = (live ? p.Hbuf : p.Hsink) + off;
#pragma unroll
                for (int j = 0; j < MG; ++j) {
                    const f32x16 v = acc[i][j];
                    u32x4 lo, hi;
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        lo[t] = pack_f16x2(v[2 * t], v[2 * t + 1]);
                        hi[t] = pack_f16x2(v[8 + 2 * t], v[9 + 2 * t]);
                    }
                    st16(ha + 32 * j, lo);
                    st16(ha + 32 * j + 8, hi);
                }
            }
        } else if constexpr (EPI == kEpiDa) {
            // A row group's loads (a, the pair weight) are all issued before
            // its first store: the wave's memory counter retires loads and
            // stores in order, so a load issued after a store would also wait
            // for that store. Unused rows go to the sink row of each buffer
            // (one address formula for every lane). The lane's row and column
            // offsets are derived here from an opaque copy of the lane index,
            // so they are not kept in registers through the stage loop.
            int ln = lane;
            asm volatile("" : "+v"(ln));
            const int elr = ln & 31, elh = ln >> 5;
#pragma unroll
            for (int i = 0; i < RG; ++i) {
                const int r = wm * (TM / 4) + i * 32 + elr;
                const bool live = r < nrows;
                const int pr = live ? rows[(par * 2 + 1) * TM + r] : p.sink_row;
                const size_t off = (size_t)pr * p.H + (size_t)c * M + wn * (M / 2) + 16 * elh;
                u16* const hw = p.Hbuf + off;
                u16* const hg = p.Gbuf + off;
                const float w = live ? p.pw[pr] : 0.f;
                u32x4 a4[MG][2];
#pragma unroll
                for (int j = 0; j < MG; ++j) {
                    a4[j][0] = ld16(hw + 32 * j);
                    a4[j][1] = ld16(hw + 32 * j + 8);
                }
                float dc = 0.f;
#pragma unroll
                for (int j = 0; j < MG; ++j) {
                    const f32x16 v = acc[i][j];
                    u32x4 wo[2], dq[2];
#pragma unroll
                    for (int h = 0; h < 2; ++h)
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            float a0, a1, e0, e1, g0, g1;
                            unpack_f16x2(a4[j][h][t], a0, a1);
                            gelu_exp2poly_grad(a0, e0, g0);
                            gelu_exp2poly_grad(a1, e1, g1);
                            const float v0 = v[8 * h + 2 * t], v1 = v[8 * h + 2 * t + 1];
                            dc = fmaf(e0, v0, dc);
                            dc = fmaf(e1, v1, dc);
                            wo[h][t] = pack_bf16x2(w * e0, w * e1);
                            dq[h][t] = pack_bf16x2(w * v0 * g0, w * v1 * g1);
                        }
                    st16(hw + 32 * j, wo[0]);
                    st16(hw + 32 * j + 8, wo[1]);
                    st16(hg + 32 * j, dq[0]);
                    st16(hg + 32 * j + 8, dq[1]);
                }
                // lanes l and l + 32 hold the two 16-column halves of a row
                dc += __shfl_xor(dc, 32);
                if (elh == 0) p.dcp[((size_t)pr * p.B + c) * 2 + wn] = dc;
            }
        } else
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int r = wm * (TM / 4) + i * 32 + lr;
            u16* dst = (r < nrows) ? p.Hbuf + (size_t)rows[(par * 2 + 1) * TM + r] * p.H + (size_t)c * M : p.Hsink;
            dst += wn * (M / 2) + 16 * lh;
#pragma unroll
            for (int j = 0; j < MG; ++j) {
                f32x16 v = acc[i][j];
                if constexpr (EPI == kEpiGeluBias) {
                    // b1 of the lane's 16 columns (Eq. block-expert-output
                    // with the FFN's first bias). The compiler's wait for
                    // these loads also covers the copies in flight: an
                    // over-wait, never an early one.
                    const float* bb = p.b_up + (size_t)(sl / p.B) * p.H + (size_t)c * M + wn * (M / 2) + 16 * lh + 32 * j;
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const f32x4 b4 = *reinterpret_cast<const f32x4*>(bb + 4 * u);
#pragma unroll
                        for (int q = 0; q < 4; ++q) v[4 * u + q] += b4[q];
                    }
                }
                u32x4 lo, hi;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    lo[t] = pack_f16x2(gelu_exp2poly(v[2 * t]), gelu_exp2poly(v[2 * t + 1]));
                    hi[t] = pack_f16x2(gelu_exp2poly(v[8 + 2 * t]), gelu_exp2poly(v[9 + 2 * t]));
                }
                st16(dst + 32 * j, lo);
                st16(dst + 32 * j + 8, hi);
            }
        }
        if (!has_next) break;
        tile = next;
        next = tq.lo + __builtin_amdgcn_readfirstlane(ctl[2]);
        info = next_info;
        par ^= 1;
        after_epi = true;
    }
    // The re-reads issued past the last tile land in LDS: let them finish
    // before the workgroup's LDS is released.
    wait_vmcnt<0>();
}

// Down-projection on the same engine as the up kernel (two stage slots,
// fragments read one k step ahead, pipelined across tiles). The 8 waves sit
// WM x (8 / WM); a tile is TM = 64 WM consecutive pairs of one expert x
// BN = (8 / WM) NG 32 output columns (wide tiles read each pair's H row for
// fewer column tiles, tall ones each weight slab for fewer rows); its stages walk the
// blocks of the tile's mask union, M/64 stages per block. A row whose mask
// lacks the stage's block reads the zero page, and a 32-row MFMA group whose
// rows all lack it skips its MFMAs. Tiles are padded to at least 4 stages
// with empty stages (no MFMAs).
template <int WM, int NG, bool F16 = true>
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void down_kernel(DownParams p) {
    using S = Stage;
    constexpr int RB = S::RB, KS = S::KSTEPS, NWV = kFfnWaves;
    constexpr int WN = NWV / WM;
    constexpr int TM = WM * 64;
    constexpr int BN = WN * NG * 32;                  // NG 32-column groups per wave
    constexpr int RG = 2;                             // 32-row groups per wave
    constexpr int LA = TM / S::ROWS_PER_DMA / NWV;
    constexpr int LB = BN / S::ROWS_PER_DMA / NWV;
    constexpr int L = LA + LB;
    constexpr int NEPI = RG * NG * 4;                 // epilogue stores per wave (fp32 rows)
    constexpr int A_BYTES = TM * RB, STAGE = (TM + BN) * RB, RING = 2 * STAGE;
    constexpr int NFETCH = 1;                         // 4-byte copies per wave for a tile's row masks
    constexpr int NR = RG + NG;
    static_assert(LA >= 1 && LB >= 1, "tile too small for one copy per wave");
    static_assert(TM % 32 == 0 && TM / 4 <= 64, "row masks: one 4-byte copy per wave");
    static_assert(NEPI + NFETCH + L < 64, "vmcnt range");
    extern __shared__ __attribute__((aligned(16))) char lds_dn[];
    uint64_t* rmask = reinterpret_cast<uint64_t*>(lds_dn + RING);   // [2][TM]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WN, wn = wave % WN;
    const int kcpb = p.M / S::SK;   // stages per block
    const TileQueue tq(p.queue, p.slices);
    // ctl as in the up kernel.
    int* ctl = reinterpret_cast<int*>(lds_dn + RING + 16 * TM);
    if (tid == 0) {
        const int t = tq.take(2);
        ctl[0] = t;
        ctl[1] = t + 1;
    }
    __syncthreads();
    int tile = tq.lo + __builtin_amdgcn_readfirstlane(ctl[0]);
    int next = tq.lo + __builtin_amdgcn_readfirstlane(ctl[1]);
    if (tile >= tq.hi) return;
    int taken = 0;

    const int lr = lane & 31, lh = lane >> 5;
    uint32_t fx[KS], fw[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) {
        fx[k] = S::off(wm * 64 + lr, 2 * k + lh);
        fw[k] = A_BYTES + S::off(wn * (BN / WN) + lr, 2 * k + lh);
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

    // Uniform description of a tile: tiles are listed row tile by row tile
    // (the column tiles of one row tile run side by side on one XCD and
    // share its H rows in L2), row tiles expert by expert; gm[i]: the block
    // mask of this wave's 32-row group i, all: the tile's.
    // With nsplit > 1, tile t is part t % nsplit of row-and-column tile
    // t / nsplit: the blocks c of the union with c % nsplit equal to the
    // part, in order, written to that part's row buffer (the merge adds the
    // parts in order). A row's part sums then cover a fixed set of its own
    // blocks, whichever rows share its tile (the order of pairs inside a
    // mask-key bin follows the arrival of atomics), so the result does not
    // depend on the tile's composition.
    struct Desc {
        int p0, nrows, e, ct, nst, nreal, sp;
        uint64_t all, gm[RG];
    };
    auto describe = [&](int t) {
        Desc D;
        const int tt = t / p.nsplit;
        D.sp = t - tt * p.nsplit;
        const int rt = tt / p.ncol;
        D.ct = tt - rt * p.ncol;
        const int* inf = reinterpret_cast<const int*>(p.rt_info + rt);
        D.p0 = ld_uniform(inf);
        D.nrows = ld_uniform(inf + 1);
        D.e = ld_uniform(inf + 2);
        const uint64_t* ms = p.rt_masks + (size_t)rt * (TM / 32 + 1);
        D.all = ld_uniform64(ms + TM / 32);
        if (p.nsplit > 1) {
            uint64_t keep = 0;
            for (int c = D.sp; c < 64; c += p.nsplit) keep |= 1ull << c;
            D.all &= keep;
        }
#pragma unroll
        for (int i = 0; i < RG; ++i) D.gm[i] = ld_uniform64(ms + wm * RG + i);
        D.nreal = __popcll(D.all) * kcpb;
        D.nst = max(D.nreal, 4);
        return D;
    };
    // A tile's row masks (TM u64): each wave copies TM bytes in 4-byte
    // pieces (a tile's first pair can be any index).
    auto fetch_masks = [&](Desc D, int par) {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(p.pair_mask + D.p0);
        if (lane < TM / 4) dma4(src + wave * (TM / 4) + lane, rmask + par * TM + wave * (TM / 8));
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
        // behind the fragment reads of a k step.
        wait_lgkmcnt0();
        wtile = wdn + ((size_t)D.e * p.d + (size_t)D.ct * BN) * hrow;
        rem_w = D.all;
        kc_w = 0;
        set_block_w();
    };
    // The copies of one stage: copy q < LA fills H rows, the rest weight rows.
    auto issue_one = [&](uint32_t slot, int q) {
        char* base = lds_dn + slot;
        if (q < LA) dma16(pa[q], base + (wave * LA + q) * 1024);
        else dma16(pb + voffB[q - LA], base + A_BYTES + (wave * LB + q - LA) * 1024);
    };
    auto issue_end = [&]() {
#pragma unroll
        for (int q = 0; q < LA; ++q) pa[q] += sa[q];
        pb += RB;
        if (++kc_w == kcpb) {
            kc_w = 0;
            rem_w &= rem_w - 1;
            set_block_w();
        }
    };
    u32x4 fxa[RG], fwa[NG], fxb[RG], fwb[NG];
    auto read_one = [&](uint32_t slot, int k, int r, u32x4 (&X)[RG], u32x4 (&W)[NG]) {
        const char* st = lds_dn + slot;
        if (r < NG) W[r] = ld16(st + fw[k] + r * 32 * RB);
        else X[r - NG] = ld16(st + fx[k] + (r - NG) * 32 * RB);
    };
    f32x16 acc[RG][NG];

    int par = 0;
    Desc cur = describe(tile);
    fetch_masks(cur, 0);
    wait_vmcnt<0>();
    __syncthreads();
    issue_tile(cur, 0);
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
        for (int q = 0; q < L; ++q) issue_one(st * STAGE, q);
        issue_end();
    }
    wait_vmcnt<L>();
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int r = 0; r < NR; ++r) read_one(0, 0, r, fxa, fwa);
    uint32_t slot = 0;
    bool after_epi = false;
    for (;;) {
        const bool has_next = next < tq.hi;
        Desc nxt;
        if (has_next) nxt = describe(next);
        // No scalar load may be in flight in the stage loop (see up_kernel).
        wait_lgkmcnt0();
#pragma unroll
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int j = 0; j < NG; ++j) acc[i][j] = f32x16{};
        // Read side: which of this wave's row groups use the block of the
        // stage being computed (bit i: group i), and the stage within it.
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
        for (int s = 0; s < nst; ++s) {
            const uint32_t other = slot ^ STAGE;
            auto kstep = [&](int k, u32x4 (&X)[RG], u32x4 (&W)[NG], u32x4 (&X2)[RG], u32x4 (&W2)[NG]) {
                const uint32_t rslot = (k == KS - 1) ? other : slot;
                const int rk = (k == KS - 1) ? 0 : k + 1;
#pragma unroll
                for (int r = 0; r < NR; ++r) read_one(rslot, rk, r, X2, W2);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < RG; ++i) {
                    if (gset & (1u << i)) {
#pragma unroll
                        for (int j = 0; j < NG; ++j)
                            acc[i][j] = F16 ? mfma32x32x16_f16(as_f16x8(W[j]), as_f16x8(X[i]), acc[i][j])
                                            : mfma32x32x16(as_bf16x8(W[j]), as_bf16x8(X[i]), acc[i][j]);
                    }
                    if (k == KS - 1) {
#pragma unroll
                        for (int q = 0; q < L; ++q)
                            if (q * RG / L == i) issue_one(slot, q);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            };
            kstep(0, fxa, fwa, fxb, fwb);
            kstep(1, fxb, fwb, fxa, fwa);
            kstep(2, fxa, fwa, fxb, fwb);
            wait_lgkmcnt0();
            wait_stage<NEPI, NFETCH>(s, after_epi, has_next);
            __builtin_amdgcn_s_barrier();
            if (s == 0 && has_next && tid == 0) taken = tq.take(1);
            if (s == 1 && has_next && tid == 0) ctl[2] = taken;
            if (s + 2 == nst) {
                // The stages issued from here on belong to the next tile (or,
                // past the last tile, re-read this tile's first stages). Its
                // row masks were copied at stage 0 and waited for at the
                // barrier of stage 2 (s >= 2 here).
                Desc D = cur;
                if (has_next) D = nxt;
                issue_tile(D, has_next ? par ^ 1 : par);
            }
            kstep(3, fxb, fwb, fxa, fwa);
            issue_end();
            if (s == 0 && has_next) fetch_masks(nxt, par ^ 1);
            if (++kc_r == kcpb) {
                kc_r = 0;
                rem_r &= rem_r - 1;
                gset = groups();
            }
            slot = other;
        }
        // Per-expert rows in fp32 (the combine weighs and sums them in fp32
        // and rounds once); lane stores 16 consecutive columns of its row
        // per 32-column group.
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int r = wm * 64 + i * 32 + lr;
            float* dst = (r < cur.nrows) ? p.part + cur.sp * p.split_stride + (size_t)(cur.p0 + r) * p.d + (size_t)cur.ct * BN
                                         : p.part_sink;
            dst += wn * (BN / WN) + 16 * lh;
#pragma unroll
            for (int j = 0; j < NG; ++j) {
                const f32x16 v = acc[i][j];
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    st16(dst + 32 * j + 4 * t, u32x4{__float_as_uint(v[4 * t]), __float_as_uint(v[4 * t + 1]),
                                                     __float_as_uint(v[4 * t + 2]), __float_as_uint(v[4 * t + 3])});
            }
        }
        if (!has_next) break;
        tile = next;
        next = tq.lo + __builtin_amdgcn_readfirstlane(ctl[2]);
        cur = nxt;
        par ^= 1;
        after_epi = true;
    }
    // The re-reads issued past the last tile land in LDS: let them finish
    // before the workgroup's LDS is released.
    wait_vmcnt<0>();
}

}  // namespace unifmoe
