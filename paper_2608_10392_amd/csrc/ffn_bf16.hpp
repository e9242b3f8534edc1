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
// mask lacks a block load zeros, and each 16-row MFMA group skips the blocks
// none of its rows use. Pairs are sorted by mask key, so tiles hold similar
// masks.
//
// Engine shared by both: 4 waves in a 2 x 2 arrangement, each wave owning a
// 128-row slab of the macro tile (8 MFMA row groups), so one B fragment read
// from LDS feeds 8 MFMAs. K is staged 64 deep through double-buffered LDS
// (row stride 72 bf16 = 144 B, conflict-free 16-byte fragment reads); the
// next stage's global loads are issued into registers before the current
// stage's MFMAs and stored to the other buffer after them, one barrier per
// stage. Both kernels are persistent over a device-built tile table, with
// consecutive tiles mapped to workgroups of the same XCD (workgroups are
// dispatched round-robin over the 8 XCDs), so co-running tiles share weight
// slabs in that XCD's L2.
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kTM = 256;          // rows (pairs) per macro tile
constexpr int kBK = 64;           // contraction depth per LDS stage
constexpr int kLdk = kBK + 8;     // padded LDS row stride (bf16 elements)
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
    float* part;
    const int* seg_off;
    const int* down_tile_off;
    const int* totals;
    const uint64_t* pair_mask;
};

// LDS elements (bf16) of the two kernels: two stages, reused by the epilogue.
__host__ __device__ constexpr int up_lds_elems(int M) {
    return 2 * (kTM + M) * kLdk > kTM * (M + 8) ? 2 * (kTM + M) * kLdk : kTM * (M + 8);
}
__host__ __device__ constexpr int down_lds_elems(int BN) { return 2 * (kTM + BN) * kLdk; }

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

template <int MW>  // M = 32 MW; each wave covers 128 rows x M / 2 columns
__global__ __launch_bounds__(kFfnThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void up_kernel(UpParams p) {
    constexpr int M = MW * 32;
    constexpr int A_ELEMS = kTM * kLdk;
    constexpr int STAGE = (kTM + M) * kLdk;
    constexpr int A_LD = kTM * 8 / kFfnThreads;   // 16-byte chunks per thread per stage
    constexpr int B_LD = M * 8 / kFfnThreads;
    extern __shared__ __attribute__((aligned(16))) u16 lds_up[];
    __shared__ int row_pair[kTM], row_tok[kTM];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int frag_r = lane & 15, frag_k = (lane >> 4) * 8;
    const int ld_r = tid >> 3, ld_c = (tid & 7) * 8;   // this thread's row / column in a stage
    const int n_tiles = p.totals[1];
    const int nk = p.d / kBK;
    for (int round = 0; round * (int)gridDim.x < n_tiles; ++round) {
        const int tile = xcd_tile(round);
        if (tile >= n_tiles) continue;
        const int s = upper_index(p.up_tile_off, p.nslab, tile);
        const int e = s / p.B, c = s - e * p.B;
        const int r0 = (tile - p.up_tile_off[s]) * kTM;
        const int nrows = min(kTM, p.slab_count[s] - r0);
        __syncthreads();
        {
            int pr = -1, tk = -1;
            if (tid < nrows) {
                pr = p.slab_rows[p.slab_off[s] + r0 + tid];
                tk = p.pair_token[pr];
            }
            row_pair[tid] = pr;
            row_tok[tid] = tk;
        }
        __syncthreads();
        const u16* W = p.Wup + ((size_t)e * p.H + (size_t)c * M) * p.d;
        int arow[A_LD];   // element offset of this thread's token rows, -1 for padding
#pragma unroll
        for (int i = 0; i < A_LD; ++i) {
            const int tk = row_tok[ld_r + 32 * i];
            arow[i] = tk >= 0 ? tk * p.d + ld_c : -1;
        }
        u32x4 ra[A_LD], rb[B_LD];
        auto gload = [&](int k0) {
#pragma unroll
            for (int i = 0; i < A_LD; ++i) {
                ra[i] = u32x4{0u, 0u, 0u, 0u};
                if (arow[i] >= 0) ra[i] = ld16(p.X + (unsigned)arow[i] + k0);
            }
#pragma unroll
            for (int i = 0; i < B_LD; ++i) rb[i] = ld16(W + (size_t)(ld_r + 32 * i) * p.d + k0 + ld_c);
        };
        auto sstore = [&](int buf) {
            u16* As = lds_up + buf * STAGE;
            u16* Bs = As + A_ELEMS;
#pragma unroll
            for (int i = 0; i < A_LD; ++i) st16(As + (ld_r + 32 * i) * kLdk + ld_c, ra[i]);
#pragma unroll
            for (int i = 0; i < B_LD; ++i) st16(Bs + (ld_r + 32 * i) * kLdk + ld_c, rb[i]);
        };
        f32x4 acc[8][MW];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        gload(0);
        sstore(0);
        __syncthreads();
        for (int ks = 0; ks < nk; ++ks) {
            const int buf = ks & 1;
            if (ks + 1 < nk) gload((ks + 1) * kBK);
            const u16* As = lds_up + buf * STAGE;
            const u16* Bs = As + A_ELEMS;
#pragma unroll
            for (int kk = 0; kk < kBK; kk += 32) {
                bf16x8 bw[MW];
#pragma unroll
                for (int j = 0; j < MW; ++j)
                    bw[j] = as_bf16x8(ld16(Bs + (wn * (M / 2) + j * 16 + frag_r) * kLdk + kk + frag_k));
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const bf16x8 af = as_bf16x8(ld16(As + (wm * 128 + i * 16 + frag_r) * kLdk + kk + frag_k));
#pragma unroll
                    for (int j = 0; j < MW; ++j) acc[i][j] = mfma16x16x32(af, bw[j], acc[i][j]);
                }
            }
            if (ks + 1 < nk) sstore(buf ^ 1);
            __syncthreads();
        }
        // GELU, round to bf16, stage the tile in LDS, store whole rows.
        constexpr int OST = M + 8;
        u16* Os = lds_up;
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = wm * 128 + i * 16 + (lane >> 4) * 4 + r;
                    const int col = wn * (M / 2) + j * 16 + (lane & 15);
                    Os[row * OST + col] = f2bf(gelu_erf(acc[i][j][r]));
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
    constexpr int A_ELEMS = kTM * kLdk;
    constexpr int STAGE = (kTM + BN) * kLdk;
    constexpr int A_LD = kTM * 8 / kFfnThreads;
    constexpr int B_LD = BN * 8 / kFfnThreads;
    extern __shared__ __attribute__((aligned(16))) u16 lds_dn[];
    __shared__ uint64_t row_mask[kTM];
    __shared__ uint64_t sub_mask[kTM / 16];
    __shared__ int blist[64];
    __shared__ int nblocks;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int frag_r = lane & 15, frag_k = (lane >> 4) * 8;
    const int ld_r = tid >> 3, ld_c = (tid & 7) * 8;
    const int ncol = p.d / BN;
    const int kc_per_block = p.M / kBK;
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
            for (int c = 0; c < p.B; ++c)
                if ((m >> c) & 1ull) blist[n++] = c;
            nblocks = n;
        }
        __syncthreads();
        uint64_t wsub[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) wsub[i] = sub_mask[wm * 8 + i];
        const u16* A0 = p.Hbuf + (size_t)(p0 + ld_r) * p.H + ld_c;
        const u16* W = p.Wdown + (size_t)e * p.d * p.H + (size_t)n0 * p.H + ld_c;
        const int nstage = nblocks * kc_per_block;
        u32x4 ra[A_LD], rb[B_LD];
        auto gload = [&](int st) {
            const int c = blist[st / kc_per_block];
            const int col = c * p.M + (st % kc_per_block) * kBK;
#pragma unroll
            for (int i = 0; i < A_LD; ++i) {
                ra[i] = u32x4{0u, 0u, 0u, 0u};
                if ((row_mask[ld_r + 32 * i] >> c) & 1ull) ra[i] = ld16(A0 + (size_t)(32 * i) * p.H + col);
            }
#pragma unroll
            for (int i = 0; i < B_LD; ++i) rb[i] = ld16(W + (size_t)(ld_r + 32 * i) * p.H + col);
        };
        auto sstore = [&](int buf) {
            u16* As = lds_dn + buf * STAGE;
            u16* Bs = As + A_ELEMS;
#pragma unroll
            for (int i = 0; i < A_LD; ++i) st16(As + (ld_r + 32 * i) * kLdk + ld_c, ra[i]);
#pragma unroll
            for (int i = 0; i < B_LD; ++i) st16(Bs + (ld_r + 32 * i) * kLdk + ld_c, rb[i]);
        };
        f32x4 acc[8][NW];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < NW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (nstage > 0) {
            gload(0);
            sstore(0);
        }
        __syncthreads();
        for (int st = 0; st < nstage; ++st) {
            const int buf = st & 1;
            const int c = blist[st / kc_per_block];
            if (st + 1 < nstage) gload(st + 1);
            const u16* As = lds_dn + buf * STAGE;
            const u16* Bs = As + A_ELEMS;
#pragma unroll
            for (int kk = 0; kk < kBK; kk += 32) {
                bf16x8 bw[NW];
#pragma unroll
                for (int j = 0; j < NW; ++j)
                    bw[j] = as_bf16x8(ld16(Bs + (wn * (BN / 2) + j * 16 + frag_r) * kLdk + kk + frag_k));
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    if ((wsub[i] >> c) & 1ull) {
                        const bf16x8 af =
                            as_bf16x8(ld16(As + (wm * 128 + i * 16 + frag_r) * kLdk + kk + frag_k));
#pragma unroll
                        for (int j = 0; j < NW; ++j) acc[i][j] = mfma16x16x32(af, bw[j], acc[i][j]);
                    }
                }
            }
            if (st + 1 < nstage) sstore(buf ^ 1);
            __syncthreads();
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
