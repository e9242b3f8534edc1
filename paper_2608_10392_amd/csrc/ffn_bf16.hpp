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
//  * 4 waves in a 2 x 2 arrangement; each wave owns TM/2 rows of the tile
//    (TM/32 MFMA row groups of v_mfma_f32_16x16x32_bf16).
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
//  * Tiles can be sized so that two workgroups share a CU (OCC = 2): while
//    one waits on a barrier or runs its epilogue, the other keeps the matrix
//    cores busy.
//  * Persistent over a device-built tile table, with consecutive tiles mapped
//    to workgroups of the same XCD (dispatch is round-robin over 8 XCDs), so
//    co-running tiles share weight slabs in that XCD's L2.
#pragma once
#include "common.hpp"

namespace unifmoe {

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

// Dynamic LDS bytes of the two kernels (ring; for up also the bf16
// epilogue tile, which reuses the ring).
__host__ __device__ constexpr int up_lds_bytes(int TM, int M, int RB, int NST) {
    return NST * (TM + M) * RB > TM * (M + 8) * 2 ? NST * (TM + M) * RB : TM * (M + 8) * 2;
}
__host__ __device__ constexpr int down_lds_bytes(int TM, int BN, int RB, int NST) { return NST * (TM + BN) * RB; }

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

template <int MW, int TM, int RB, int NST, int OCC>
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void up_kernel(UpParams p) {
    using S = Stage<RB>;
    constexpr int M = MW * 32;
    constexpr int RG = TM / 32;                       // MFMA row groups per wave
    constexpr int LA = TM / S::ROWS_PER_DMA / 4;      // A DMA instructions per wave per stage
    constexpr int LB = M / S::ROWS_PER_DMA / 4;       // B DMA instructions per wave per stage
    constexpr int A_BYTES = TM * RB, STAGE = (TM + M) * RB;
    static_assert(LA >= 1 && LB >= 1, "tile too small for one DMA per wave");
    extern __shared__ __attribute__((aligned(16))) char lds_up[];
    __shared__ int row_pair[TM], row_tok[TM];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int n_tiles = p.totals[1];
    const int nk = p.d / S::SK;
    for (int round = 0; round * (int)gridDim.x < n_tiles; ++round) {
        const int tile = xcd_tile(round);
        if (tile >= n_tiles) continue;
        const int s = upper_index(p.up_tile_off, p.nslab, tile);
        const int e = s / p.B, c = s - e * p.B;
        const int r0 = (tile - p.up_tile_off[s]) * TM;
        const int nrows = min(TM, p.slab_count[s] - r0);
        wait_vmcnt<0>();          // previous tile's stores are done
        __syncthreads();
        for (int t = tid; t < TM; t += kFfnThreads) {
            int pr = -1, tk = 0;  // rows past the slab read token 0; never stored
            if (t < nrows) {
                pr = p.slab_rows[p.slab_off[s] + r0 + t];
                tk = p.pair_token[pr];
            }
            row_pair[t] = pr;
            row_tok[t] = tk;
        }
        __syncthreads();
        // Per-lane global sources of this wave's DMA instructions (k0 = 0).
        const u16* srcA[LA];
        const u16* srcB[LB];
        const u16* W = p.Wup + ((size_t)e * p.H + (size_t)c * M) * p.d;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            int r, ch;
            S::slot((wave * LA + j) * S::ROWS_PER_DMA, lane, r, ch);
            srcA[j] = p.X + (size_t)row_tok[r] * p.d + ch * 8;
        }
#pragma unroll
        for (int j = 0; j < LB; ++j) {
            int r, ch;
            S::slot((wave * LB + j) * S::ROWS_PER_DMA, lane, r, ch);
            srcB[j] = W + (size_t)r * p.d + ch * 8;
        }
        auto issue = [&](int st) {
            char* base = lds_up + (st % NST) * STAGE;
            const int k0 = st * S::SK;
#pragma unroll
            for (int j = 0; j < LA; ++j) dma16(srcA[j] + k0, base + (wave * LA + j) * 1024);
#pragma unroll
            for (int j = 0; j < LB; ++j) dma16(srcB[j] + k0, base + A_BYTES + (wave * LB + j) * 1024);
        };
        f32x4 acc[RG][MW];
#pragma unroll
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int st = 0; st < NST - 1 && st < nk; ++st) issue(st);
        for (int st = 0; st < nk; ++st) {
            stage_ready<LA + LB, NST>(st, nk);
            if (st + NST - 1 < nk) issue(st + NST - 1);
            const char* As = lds_up + (st % NST) * STAGE;
            const char* Bs = As + A_BYTES;
#pragma unroll
            for (int kk = 0; kk < S::KSTEPS; ++kk) {
                bf16x8 bw[MW];
#pragma unroll
                for (int j = 0; j < MW; ++j)
                    bw[j] = as_bf16x8(ld16(Bs + S::off(wn * (M / 2) + j * 16 + (lane & 15), kk * 4 + (lane >> 4))));
#pragma unroll
                for (int i = 0; i < RG; ++i) {
                    const bf16x8 af = as_bf16x8(
                        ld16(As + S::off(wm * (TM / 2) + i * 16 + (lane & 15), kk * 4 + (lane >> 4))));
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
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = wm * (TM / 2) + i * 16 + (lane >> 4) * 4 + r;
                    const int col = wn * (M / 2) + j * 16 + (lane & 15);
                    Os[row * OST + col] = f2bf(gelu_as7126(acc[i][j][r]));
                }
        __syncthreads();
        for (int i = tid; i < TM * (M / 8); i += kFfnThreads) {
            const int r = i / (M / 8), ch = i - (i / (M / 8)) * (M / 8);
            const int pr = row_pair[r];
            if (pr >= 0)
                st16(p.Hbuf + (size_t)pr * p.H + (size_t)c * M + ch * 8, ld16(Os + r * OST + ch * 8));
        }
    }
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
            srcB[j] = W + (size_t)r * p.H + ch * 8;
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
                        for (int j = 0; j < NW; ++j) acc[i][j] = mfma16x16x32(af, bw[j], acc[i][j]);
                    }
                }
            }
            wait_lgkmcnt0();
        }
        // fp32 per-expert rows; each 16-lane group writes 64 contiguous bytes.
#pragma unroll
        for (int i = 0; i < RG; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = wm * (TM / 2) + i * 16 + (lane >> 4) * 4 + r;
                if (row < nrows) {
                    float* dst = p.part + (size_t)(p0 + row) * p.d + n0 + wn * (BN / 2) + (lane & 15);
#pragma unroll
                    for (int j = 0; j < NW; ++j) dst[j * 16] = acc[i][j][r];
                }
            }
    }
}

}  // namespace unifmoe
