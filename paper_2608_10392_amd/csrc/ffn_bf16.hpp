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
    uint32_t x_bytes, w_bytes;   // sizes of X and W_up (each below 4 GiB)
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
    int d, M, B, H, K1;
    const u16* Hbuf;
    const u16* Wdown;
    const u16* zero16;   // 16 zero bytes in device memory
    float* part;
    const int* seg_off;
    const int* down_tile_off;
    const int* totals;
    const uint64_t* pair_mask;
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

// Dynamic LDS bytes of the two kernels: the stage ring; for up also the
// row lists (tokens, pairs) of the current and the next tile.
__host__ __device__ constexpr int up_lds_bytes(int TM, int M, int RB, int NST) { return NST * (TM + M) * RB + 16 * TM; }
__host__ __device__ constexpr int down_lds_bytes(int TM, int BN, int RB, int NST) { return NST * (TM + BN) * RB; }

// Tile handled by this workgroup in persistent round `round`: a contiguous
// range of tiles per XCD. gridDim.x is a multiple of kXcds.
__device__ __forceinline__ int xcd_tile(int round) {
    const int per = gridDim.x / kXcds;
    return round * gridDim.x + (blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
}

// Wait for stage s of n given that stages up to min(n-1, s+NST-2) were
// issued, L loads per stage per wave; then make it visible to all waves.
template <int L, int NST>
__device__ __forceinline__ void stage_ready(int s, int n) {
    const int ahead = min(n - 1 - s, NST - 2);
    if (NST >= 4 && ahead >= 2) wait_vmcnt<(NST >= 4 ? 2 * L : 0)>();
    else if (NST >= 3 && ahead >= 1) wait_vmcnt<(NST >= 3 ? L : 0)>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
}

// Wait until at most n vector-memory operations of this wave are pending,
// for the few counts the GEMM pipelines use (anything else waits for all).
template <int L, int E>
__device__ __forceinline__ void wait_vm_after(int n) {
    if (n == L) wait_vmcnt<L>();
    else if (n == L + 1) wait_vmcnt<L + 1>();
    else if (n == L + E) wait_vmcnt<L + E>();
    else if (n == L + E + 1) wait_vmcnt<L + E + 1>();
    else if (n == E) wait_vmcnt<E>();
    else if (n == E + 1) wait_vmcnt<E + 1>();
    else if (n == 1) wait_vmcnt<1>();
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
    static_assert(L + NEPI + 1 < 64, "vmcnt range");
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
    // Copy sources: buffer loads with per-lane offsets fixed for a tile and
    // the k position (and the weight slab) in the scalar offset. Token rows
    // past the tile's count read zeros.
    const uint32_t row_bytes = (uint32_t)p.d * 2;
    const rsrc_t xr = make_rsrc(p.X, p.x_bytes);
    const rsrc_t wr = make_rsrc(p.Wup, p.w_bytes);
    uint32_t voffB[LB];
#pragma unroll
    for (int j = 0; j < LB; ++j) {
        int r, ch;
        S::slot((wave * LB + j) * S::ROWS_PER_DMA, lane, r, ch);
        voffB[j] = (uint32_t)group_col(r >> 4, r & 15) * row_bytes + ch * 16;
    }
    uint32_t voffA[LA];   // token rows of the tile being issued
    uint32_t wslab = 0;   // byte offset of that tile's weight slab

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
        wslab = ((uint32_t)e * (uint32_t)p.H + (uint32_t)c * M) * row_bytes;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            int r, ch;
            S::slot((wave * LA + j) * S::ROWS_PER_DMA, lane, r, ch);
            voffA[j] = (r < nrows) ? (uint32_t)rows[par * 2 * TM + r] * row_bytes + ch * 16 : kOutOfRange;
        }
    };
    // Ring slots of the next stage to issue and of the next stage to read,
    // and the k offset (bytes) of the next stage to issue.
    int slot_w = 0, slot_r = 0;
    uint32_t k_w = 0;
    int issued = 0;
    auto issue = [&]() {
        char* base = lds_up + slot_w * STAGE;
#pragma unroll
        for (int j = 0; j < LA; ++j) dma16(xr, voffA[j], k_w, base + (wave * LA + j) * 1024);
#pragma unroll
        for (int j = 0; j < LB; ++j) dma16(wr, voffB[j], wslab + k_w, base + A_BYTES + (wave * LB + j) * 1024);
        slot_w = (slot_w == NST - 1) ? 0 : slot_w + 1;
        k_w += S::SK * 2;
        ++issued;
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
                const int n_after = L + (after_epi ? NEPI : 0) + ((s == 1 && has_next) ? 1 : 0);
                wait_vm_after<L, NEPI>(n_after);
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
            issue();
            load_frags(A2, B2);
#pragma unroll
            for (int i = 0; i < RG; ++i)
#pragma unroll
                for (int j = 0; j < MW; ++j) acc[i][j] = mfma16x16x32(as_bf16x8(Bw[j]), as_bf16x8(A[i]), acc[i][j]);
            // Interleave the copies and fragment reads with the MFMAs.
#pragma unroll
            for (int q = 0; q < L; ++q) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
            }
#pragma unroll
            for (int q = L; q < RG + MW; ++q) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, RG * MW - (RG + MW > L ? RG + MW : L), 0);
            __builtin_amdgcn_sched_barrier(0);
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

template <int NW, int TM, int RB, int NST, int OCC>
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void down_kernel(DownParams p) {
    using S = Stage<RB>;
    constexpr int BN = NW * 32;
    constexpr int RG = TM / 32;
    constexpr int LA = TM / S::ROWS_PER_DMA / 4;
    constexpr int LB = BN / S::ROWS_PER_DMA / 4;
    constexpr int A_BYTES = TM * RB, STAGE = (TM + BN) * RB;
    static_assert(LA >= 1 && LB >= 1, "tile too small for one DMA per wave");
    extern __shared__ __attribute__((aligned(16))) char lds_dn[];
    __shared__ uint64_t row_mask[TM];
    __shared__ uint64_t sub_mask[TM / 16];
    __shared__ int blist[64];
    __shared__ int nblocks;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int ncol = p.d / BN;
    const int kc_per_block = p.M / S::SK;
    const int n_tiles = p.totals[2];
    for (int round = 0; round * (int)gridDim.x < n_tiles; ++round) {
        const int tile = xcd_tile(round);
        if (tile >= n_tiles) continue;
        const int e = upper_index(p.down_tile_off, p.K1, tile);
        const int local = tile - p.down_tile_off[e];
        const int rt = local / ncol, ct = local - rt * ncol;
        const int p0 = p.seg_off[e] + rt * TM;
        const int nrows = min(TM, p.seg_off[e + 1] - p0);
        const int n0 = ct * BN;
        wait_vmcnt<0>();          // previous tile's stores are done
        __syncthreads();
        for (int t = tid; t < TM; t += kFfnThreads) row_mask[t] = (t < nrows) ? p.pair_mask[p0 + t] : 0ull;
        __syncthreads();
        if (tid < TM / 16) {
            uint64_t m = 0;
            for (int r = 0; r < 16; ++r) m |= row_mask[tid * 16 + r];
            sub_mask[tid] = m;
        }
        __syncthreads();
        if (tid == 0) {
            uint64_t m = 0;
            for (int g = 0; g < TM / 16; ++g) m |= sub_mask[g];
            int n = 0;
            for (int cc = 0; cc < p.B; ++cc)
                if ((m >> cc) & 1ull) blist[n++] = cc;
            nblocks = n;
        }
        __syncthreads();
        // Block masks of this wave's 16-row groups, as scalars (wave-uniform).
        uint32_t wsub_lo[RG], wsub_hi[RG];
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const uint64_t m = sub_mask[wm * RG + i];
            wsub_lo[i] = __builtin_amdgcn_readfirstlane((uint32_t)m);
            wsub_hi[i] = __builtin_amdgcn_readfirstlane((uint32_t)(m >> 32));
        }
        // Per-lane sources: A rows are pairs p0 + r (or the zero page when the
        // row's mask lacks the stage's block), B rows are output columns n0 + r.
        const u16* srcA[LA];
        uint64_t mA[LA];
        const u16* srcB[LB];
        const u16* W = p.Wdown + ((size_t)e * p.d + n0) * p.H;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            int r, ch;
            S::slot((wave * LA + j) * S::ROWS_PER_DMA, lane, r, ch);
            srcA[j] = p.Hbuf + (size_t)(p0 + r) * p.H + ch * 8;
            mA[j] = row_mask[r];
        }
#pragma unroll
        for (int j = 0; j < LB; ++j) {
            int r, ch;
            S::slot((wave * LB + j) * S::ROWS_PER_DMA, lane, r, ch);
            srcB[j] = W + (size_t)group_col(r >> 4, r & 15) * p.H + ch * 8;
        }
        const int nst = nblocks * kc_per_block;
        auto issue = [&](int st) {
            char* base = lds_dn + (st % NST) * STAGE;
            const int cb = blist[st / kc_per_block];
            const int col = cb * p.M + (st - (st / kc_per_block) * kc_per_block) * S::SK;
#pragma unroll
            for (int j = 0; j < LA; ++j) {
                const u16* src = ((mA[j] >> cb) & 1ull) ? srcA[j] + col : p.zero16;
                dma16(src, base + (wave * LA + j) * 1024);
            }
#pragma unroll
            for (int j = 0; j < LB; ++j) dma16(srcB[j] + col, base + A_BYTES + (wave * LB + j) * 1024);
        };
        f32x4 acc[RG][NW];
#pragma unroll
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int j = 0; j < NW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int st = 0; st < NST - 1 && st < nst; ++st) issue(st);
        for (int st = 0; st < nst; ++st) {
            stage_ready<LA + LB, NST>(st, nst);
            if (st + NST - 1 < nst) issue(st + NST - 1);
            const int cb = __builtin_amdgcn_readfirstlane(blist[st / kc_per_block]);
            const char* As = lds_dn + (st % NST) * STAGE;
            const char* Bs = As + A_BYTES;
#pragma unroll
            for (int kk = 0; kk < S::KSTEPS; ++kk) {
                bf16x8 bw[NW];
#pragma unroll
                for (int j = 0; j < NW; ++j)
                    bw[j] = as_bf16x8(ld16(Bs + S::off(wn * (BN / 2) + j * 16 + (lane & 15), kk * 4 + (lane >> 4))));
#pragma unroll
                for (int i = 0; i < RG; ++i) {
                    if ((((cb < 32) ? wsub_lo[i] >> cb : wsub_hi[i] >> (cb - 32)) & 1u) != 0u) {
                        const bf16x8 af = as_bf16x8(
                            ld16(As + S::off(wm * (TM / 2) + i * 16 + (lane & 15), kk * 4 + (lane >> 4))));
#pragma unroll
                        for (int j = 0; j < NW; ++j) acc[i][j] = mfma16x16x32(bw[j], af, acc[i][j]);
                    }
                }
            }
            wait_lgkmcnt0();
        }
        // fp32 per-expert rows; lane stores 8 consecutive columns of its row.
#pragma unroll
        for (int i = 0; i < RG; ++i) {
            const int row = wm * (TM / 2) + i * 16 + (lane & 15);
            if (row >= nrows) continue;
            float* dst = p.part + (size_t)(p0 + row) * p.d + n0 + wn * (BN / 2) + 8 * (lane >> 4);
#pragma unroll
            for (int J = 0; J < NW / 2; ++J) {
                st16(dst + 32 * J, __builtin_bit_cast(u32x4, acc[i][2 * J]));
                st16(dst + 32 * J + 4, __builtin_bit_cast(u32x4, acc[i][2 * J + 1]));
            }
        }
    }
}

}  // namespace unifmoe
