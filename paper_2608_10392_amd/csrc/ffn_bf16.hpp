// Block-sparse expert FFN on the bf16 matrix cores (Eq. block-expert-output).
//
// Up-projection + GELU, one tile = 256 rows of one (expert e, block c) slab:
//   Hbuf[pair, c M .. c M + M) = GELU(X[token(pair)] K_e[:, block c])
// Rows come from the slab's compacted pair list, so no inactive (pair, block)
// is computed. The tile spans the whole block width M, so each gathered token
// row is read once per slab.
//
// Down-projection, one tile = 256 consecutive pairs of one expert segment x
// BN output columns:
//   part[pair, n] = sum over blocks c of the pair's mask of
//                   Hbuf[pair, block c] . V_e[block c, n]        (fp32)
// The contraction runs over the union of the tile's block masks; rows whose
// mask lacks a block read a zero page instead, and each 16-row MFMA group
// skips the blocks none of its rows use. Pairs are sorted by mask key, so
// tiles hold similar masks.
//
// Engine shared by both kernels:
//  * 4 waves in a 2 x 2 arrangement; each wave owns 128 rows of the macro
//    tile (8 MFMA row groups), so one B fragment read from LDS feeds 8 MFMAs.
//  * K advances 64 per stage (two v_mfma_f32_16x16x32_bf16 steps). A stage
//    holds 128-byte rows (whole cache lines); the 16-byte chunk c of row r
//    sits at slot c ^ ((r >> 1) & 7). Measured with the LDS bank-conflict
//    counter on gfx950, this makes the fragment reads (16 rows x 4 chunks per
//    instruction) conflict-free, at 4 cycles per 1 KB read; the unswizzled
//    layout and a padded 144-byte stride run at half that rate or worse.
//  * Stages are filled by global_load_lds_dwordx4 (no register staging): one
//    instruction fills 8 rows, each lane fetching the global chunk that
//    belongs in its swizzled slot. NST stages rotate (as many as LDS holds);
//    NST - 1 are in flight while one is consumed. Waits are explicit vmcnt
//    counts followed by a bare s_barrier (a __syncthreads fence would drain
//    every load).
//  * Persistent over a device-built tile table, with consecutive tiles mapped
//    to workgroups of the same XCD (dispatch is round-robin over 8 XCDs), so
//    co-running tiles share weight slabs in that XCD's L2.
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kTM = 256;          // rows (pairs) per macro tile
constexpr int kSK = 64;           // contraction depth per stage
constexpr int kRowB = kSK * 2;    // bytes per staged row (one cache line)
constexpr int kRowsPerDma = 1024 / kRowB;
constexpr int kLdsMax = 160 * 1024 - 4096;  // dynamic LDS budget (static arrays use the rest)
constexpr int kFfnThreads = 256;
constexpr int kXcds = 8;

struct UpParams {
    int d, M, B, H, nslab;
    const u16* X;
    const u16* Wup;
    u16* Hbuf;
    const int* slab_rows;
    const int* slab_off;
    const int* slab_count;
    const int* up_tile_off;
    const int* totals;
    const int* pair_token;
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

// Stages of the LDS ring for a macro tile of kTM + N rows (at most 4).
__host__ __device__ constexpr int ring_stages(int N) {
    return kLdsMax / ((kTM + N) * kRowB) < 4 ? kLdsMax / ((kTM + N) * kRowB) : 4;
}
// Dynamic LDS bytes: the stage ring, or the bf16 epilogue tile if larger.
__host__ __device__ constexpr int up_lds_bytes(int M) {
    return ring_stages(M) * (kTM + M) * kRowB > kTM * (M + 8) * 2 ? ring_stages(M) * (kTM + M) * kRowB
                                                                   : kTM * (M + 8) * 2;
}
__host__ __device__ constexpr int down_lds_bytes(int BN) { return ring_stages(BN) * (kTM + BN) * kRowB; }

// Byte offset of 16-byte chunk `c` (0..7) of row `r` inside a stage tile.
__device__ __forceinline__ int swz(int r, int c) { return r * kRowB + ((c ^ ((r >> 1) & 7)) << 4); }

// Largest i in [0, n) with off[i] <= x (off ascending, off[0] = 0 <= x).
__device__ __forceinline__ int upper_index(const int* off, int n, int x) {
    int lo = 0, hi = n;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (off[mid] <= x) lo = mid;
        else hi = mid;
    }
    return lo;
}

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

// Row r, chunk c that lane `lane` fills when one DMA instruction covers rows
// r0 .. r0 + kRowsPerDma - 1 of a stage tile.
__device__ __forceinline__ void dma_slot(int r0, int lane, int& r, int& c) {
    r = r0 + (lane >> 3);
    c = (lane & 7) ^ ((r >> 1) & 7);
}

template <int MW>  // M = 32 MW; each wave covers 128 rows x M / 2 columns
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void up_kernel(UpParams p) {
    constexpr int M = MW * 32;
    constexpr int NST = ring_stages(M);
    constexpr int LA = kTM / kRowsPerDma / 4;   // A DMA instructions per wave per stage
    constexpr int LB = M / kRowsPerDma / 4;     // B DMA instructions per wave per stage
    constexpr int A_BYTES = kTM * kRowB, STAGE = (kTM + M) * kRowB;
    extern __shared__ __attribute__((aligned(16))) char lds_up[];
    __shared__ int row_pair[kTM], row_tok[kTM];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int n_tiles = p.totals[1];
    const int nk = p.d / kSK;
    for (int round = 0; round * (int)gridDim.x < n_tiles; ++round) {
        const int tile = xcd_tile(round);
        if (tile >= n_tiles) continue;
        const int s = upper_index(p.up_tile_off, p.nslab, tile);
        const int e = s / p.B, c = s - e * p.B;
        const int r0 = (tile - p.up_tile_off[s]) * kTM;
        const int nrows = min(kTM, p.slab_count[s] - r0);
        wait_vmcnt<0>();          // previous tile's stores are done
        __syncthreads();
        {
            int pr = -1, tk = 0;  // rows past the slab read token 0; never stored
            if (tid < nrows) {
                pr = p.slab_rows[p.slab_off[s] + r0 + tid];
                tk = p.pair_token[pr];
            }
            row_pair[tid] = pr;
            row_tok[tid] = tk;
        }
        __syncthreads();
        // Per-lane global sources of this wave's DMA instructions (k0 = 0).
        const u16* srcA[LA];
        const u16* srcB[LB];
        const u16* W = p.Wup + ((size_t)e * p.H + (size_t)c * M) * p.d;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            int r, ch;
            dma_slot((wave * LA + j) * kRowsPerDma, lane, r, ch);
            srcA[j] = p.X + (size_t)row_tok[r] * p.d + ch * 8;
        }
#pragma unroll
        for (int j = 0; j < LB; ++j) {
            int r, ch;
            dma_slot((wave * LB + j) * kRowsPerDma, lane, r, ch);
            srcB[j] = W + (size_t)r * p.d + ch * 8;
        }
        auto issue = [&](int st) {
            char* base = lds_up + (st % NST) * STAGE;
            const int k0 = st * kSK;
#pragma unroll
            for (int j = 0; j < LA; ++j) dma16(srcA[j] + k0, base + (wave * LA + j) * 1024);
#pragma unroll
            for (int j = 0; j < LB; ++j) dma16(srcB[j] + k0, base + A_BYTES + (wave * LB + j) * 1024);
        };
        f32x4 acc[8][MW];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int st = 0; st < NST - 1 && st < nk; ++st) issue(st);
        for (int st = 0; st < nk; ++st) {
            stage_ready<LA + LB, NST>(st, nk);
            if (st + NST - 1 < nk) issue(st + NST - 1);
            const char* As = lds_up + (st % NST) * STAGE;
            const char* Bs = As + A_BYTES;
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                bf16x8 bw[MW];
#pragma unroll
                for (int j = 0; j < MW; ++j)
                    bw[j] = as_bf16x8(ld16(Bs + swz(wn * (M / 2) + j * 16 + (lane & 15), kk * 4 + (lane >> 4))));
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const bf16x8 af =
                        as_bf16x8(ld16(As + swz(wm * 128 + i * 16 + (lane & 15), kk * 4 + (lane >> 4))));
#pragma unroll
                    for (int j = 0; j < MW; ++j) acc[i][j] = mfma16x16x32(af, bw[j], acc[i][j]);
                }
            }
            wait_lgkmcnt0();
        }
        // GELU, round to bf16, stage the tile in LDS, store whole rows.
        __syncthreads();
        constexpr int OST = M + 8;
        u16* Os = reinterpret_cast<u16*>(lds_up);
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = wm * 128 + i * 16 + (lane >> 4) * 4 + r;
                    const int col = wn * (M / 2) + j * 16 + (lane & 15);
                    Os[row * OST + col] = f2bf(gelu_as7126(acc[i][j][r]));
                }
        __syncthreads();
        for (int i = tid; i < kTM * (M / 8); i += kFfnThreads) {
            const int r = i / (M / 8), ch = i - (i / (M / 8)) * (M / 8);
            const int pr = row_pair[r];
            if (pr >= 0)
                st16(p.Hbuf + (size_t)pr * p.H + (size_t)c * M + ch * 8, ld16(Os + r * OST + ch * 8));
        }
    }
}

template <int NW>  // BN = 32 NW output columns; each wave covers 128 rows x BN / 2
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void down_kernel(DownParams p) {
    constexpr int BN = NW * 32;
    constexpr int NST = ring_stages(BN);
    constexpr int LA = kTM / kRowsPerDma / 4;
    constexpr int LB = BN / kRowsPerDma / 4;
    constexpr int A_BYTES = kTM * kRowB, STAGE = (kTM + BN) * kRowB;
    extern __shared__ __attribute__((aligned(16))) char lds_dn[];
    __shared__ uint64_t row_mask[kTM];
    __shared__ uint64_t sub_mask[kTM / 16];
    __shared__ int blist[64];
    __shared__ int nblocks;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int ncol = p.d / BN;
    const int kc_per_block = p.M / kSK;
    const int n_tiles = p.totals[2];
    for (int round = 0; round * (int)gridDim.x < n_tiles; ++round) {
        const int tile = xcd_tile(round);
        if (tile >= n_tiles) continue;
        const int e = upper_index(p.down_tile_off, p.K1, tile);
        const int local = tile - p.down_tile_off[e];
        const int rt = local / ncol, ct = local - rt * ncol;
        const int p0 = p.seg_off[e] + rt * kTM;
        const int nrows = min(kTM, p.seg_off[e + 1] - p0);
        const int n0 = ct * BN;
        wait_vmcnt<0>();          // previous tile's stores are done
        __syncthreads();
        row_mask[tid] = (tid < nrows) ? p.pair_mask[p0 + tid] : 0ull;
        __syncthreads();
        if (tid < kTM / 16) {
            uint64_t m = 0;
            for (int r = 0; r < 16; ++r) m |= row_mask[tid * 16 + r];
            sub_mask[tid] = m;
        }
        __syncthreads();
        if (tid == 0) {
            uint64_t m = 0;
            for (int g = 0; g < kTM / 16; ++g) m |= sub_mask[g];
            int n = 0;
            for (int cc = 0; cc < p.B; ++cc)
                if ((m >> cc) & 1ull) blist[n++] = cc;
            nblocks = n;
        }
        __syncthreads();
        // Block masks of this wave's 16-row groups, as scalars (wave-uniform).
        uint32_t wsub_lo[8], wsub_hi[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint64_t m = sub_mask[wm * 8 + i];
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
            dma_slot((wave * LA + j) * kRowsPerDma, lane, r, ch);
            srcA[j] = p.Hbuf + (size_t)(p0 + r) * p.H + ch * 8;
            mA[j] = row_mask[r];
        }
#pragma unroll
        for (int j = 0; j < LB; ++j) {
            int r, ch;
            dma_slot((wave * LB + j) * kRowsPerDma, lane, r, ch);
            srcB[j] = W + (size_t)r * p.H + ch * 8;
        }
        const int nst = nblocks * kc_per_block;
        auto issue = [&](int st) {
            char* base = lds_dn + (st % NST) * STAGE;
            const int cb = blist[st / kc_per_block];
            const int col = cb * p.M + (st - (st / kc_per_block) * kc_per_block) * kSK;
#pragma unroll
            for (int j = 0; j < LA; ++j) {
                const u16* src = ((mA[j] >> cb) & 1ull) ? srcA[j] + col : p.zero16;
                dma16(src, base + (wave * LA + j) * 1024);
            }
#pragma unroll
            for (int j = 0; j < LB; ++j) dma16(srcB[j] + col, base + A_BYTES + (wave * LB + j) * 1024);
        };
        f32x4 acc[8][NW];
#pragma unroll
        for (int i = 0; i < 8; ++i)
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
            for (int kk = 0; kk < 2; ++kk) {
                bf16x8 bw[NW];
#pragma unroll
                for (int j = 0; j < NW; ++j)
                    bw[j] = as_bf16x8(ld16(Bs + swz(wn * (BN / 2) + j * 16 + (lane & 15), kk * 4 + (lane >> 4))));
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    if ((((cb < 32) ? wsub_lo[i] >> cb : wsub_hi[i] >> (cb - 32)) & 1u) != 0u) {
                        const bf16x8 af =
                            as_bf16x8(ld16(As + swz(wm * 128 + i * 16 + (lane & 15), kk * 4 + (lane >> 4))));
#pragma unroll
                        for (int j = 0; j < NW; ++j) acc[i][j] = mfma16x16x32(af, bw[j], acc[i][j]);
                    }
                }
            }
            wait_lgkmcnt0();
        }
        // fp32 per-expert rows; each 16-lane group writes 64 contiguous bytes.
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = wm * 128 + i * 16 + (lane >> 4) * 4 + r;
                if (row < nrows) {
                    float* dst = p.part + (size_t)(p0 + row) * p.d + n0 + wn * (BN / 2) + (lane & 15);
#pragma unroll
                    for (int j = 0; j < NW; ++j) dst[j * 16] = acc[i][j][r];
                }
            }
    }
}

}  // namespace unifmoe
