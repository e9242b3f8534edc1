// Block-sparse expert FFN on the bf16 matrix cores (Eq. block-expert-output).
//
// Up-projection + GELU, one tile = 128 rows of one (expert e, block c) slab:
//   Hbuf[pair, c M .. c M + M) = GELU(X[token(pair)] K_e[:, block c])
// Rows come from the slab's compacted pair list, so no inactive (pair, block)
// is computed. The tile spans the whole block width M, so each gathered token
// row is read once per slab.
//
// Down-projection, one tile = 128 consecutive pairs of one expert segment x
// 128 output columns:
//   part[pair, n] = sum over blocks c of the pair's mask of
//                   Hbuf[pair, block c] . V_e[block c, n]        (fp32)
// The contraction runs over the union of the tile's block masks; rows whose
// mask lacks a block load zeros, and each 16-row MFMA group skips the blocks
// none of its rows use. Pairs are sorted by mask key, so tiles hold similar
// masks.
//
// Both kernels are persistent: each workgroup walks a device-built tile
// table, so the host never reads counts back. 4 waves per workgroup in a
// 2 x 2 arrangement; operands staged through LDS with a padded row stride
// (72 bf16 = 144 B) so the 16-byte fragment reads are bank-conflict free.
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kBM = 128;          // rows (pairs) per tile
constexpr int kBN = 128;          // output columns per down-projection tile
constexpr int kBK = 64;           // contraction depth staged per LDS round
constexpr int kLdk = kBK + 8;     // padded LDS row stride (bf16 elements)
constexpr int kFfnThreads = 256;

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

__host__ __device__ constexpr int up_lds_elems(int M) {
    return ((kBM + M) * kLdk > kBM * (M + 8)) ? (kBM + M) * kLdk : kBM * (M + 8);
}
__host__ __device__ constexpr int down_lds_elems() { return (kBM + kBN) * kLdk; }

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

template <int MW>  // M = 32 MW; each wave covers M / 2 columns = MW tiles of 16
__global__ __launch_bounds__(kFfnThreads) void up_kernel(UpParams p) {
    constexpr int M = MW * 32;
    extern __shared__ __attribute__((aligned(16))) u16 lds_up[];
    u16* As = lds_up;
    u16* Bs = lds_up + kBM * kLdk;
    __shared__ int row_pair[kBM], row_tok[kBM];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int frag_r = lane & 15, frag_k = (lane >> 4) * 8;
    const int n_tiles = p.totals[1];
    for (int tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        const int s = upper_index(p.up_tile_off, p.nslab, tile);
        const int e = s / p.B, c = s - e * p.B;
        const int r0 = (tile - p.up_tile_off[s]) * kBM;
        const int nrows = min(kBM, p.slab_count[s] - r0);
        __syncthreads();
        if (tid < kBM) {
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
        f32x4 acc[4][MW];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < p.d; k0 += kBK) {
            for (int i = tid; i < kBM * 8; i += kFfnThreads) {
                const int r = i >> 3, ch = i & 7;
                u32x4 v = {0u, 0u, 0u, 0u};
                const int tk = row_tok[r];
                if (tk >= 0) v = ld16(p.X + (size_t)tk * p.d + k0 + ch * 8);
                st16(As + r * kLdk + ch * 8, v);
            }
            for (int i = tid; i < M * 8; i += kFfnThreads) {
                const int r = i >> 3, ch = i & 7;
                st16(Bs + r * kLdk + ch * 8, ld16(W + (size_t)r * p.d + k0 + ch * 8));
            }
            __syncthreads();
#pragma unroll
            for (int kk = 0; kk < kBK; kk += 32) {
                bf16x8 af[4], bw[MW];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    af[i] = as_bf16x8(ld16(As + (wm * 64 + i * 16 + frag_r) * kLdk + kk + frag_k));
#pragma unroll
                for (int j = 0; j < MW; ++j)
                    bw[j] = as_bf16x8(ld16(Bs + (wn * (M / 2) + j * 16 + frag_r) * kLdk + kk + frag_k));
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < MW; ++j) acc[i][j] = mfma16x16x32(af[i], bw[j], acc[i][j]);
            }
            __syncthreads();
        }
        // GELU, round to bf16, stage the tile in LDS, store whole rows.
        constexpr int OST = M + 8;
        u16* Os = lds_up;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = wm * 64 + i * 16 + (lane >> 4) * 4 + r;
                    const int col = wn * (M / 2) + j * 16 + (lane & 15);
                    Os[row * OST + col] = f2bf(gelu_erf(acc[i][j][r]));
                }
        __syncthreads();
        for (int i = tid; i < kBM * (M / 8); i += kFfnThreads) {
            const int r = i / (M / 8), ch = i - (i / (M / 8)) * (M / 8);
            const int pr = row_pair[r];
            if (pr >= 0)
                st16(p.Hbuf + (size_t)pr * p.H + (size_t)c * M + ch * 8, ld16(Os + r * OST + ch * 8));
        }
    }
}

__global__ __launch_bounds__(kFfnThreads) void down_kernel(DownParams p) {
    extern __shared__ __attribute__((aligned(16))) u16 lds_dn[];
    u16* As = lds_dn;
    u16* Bs = lds_dn + kBM * kLdk;
    __shared__ uint64_t row_mask[kBM];
    __shared__ uint64_t sub_mask[kBM / 16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int frag_r = lane & 15, frag_k = (lane >> 4) * 8;
    const int ncol = p.d / kBN;
    const int n_tiles = p.totals[2];
    for (int tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        const int e = upper_index(p.down_tile_off, p.K1, tile);
        const int local = tile - p.down_tile_off[e];
        const int rt = local / ncol, ct = local - rt * ncol;
        const int p0 = p.seg_off[e] + rt * kBM;
        const int nrows = min(kBM, p.seg_off[e + 1] - p0);
        const int n0 = ct * kBN;
        __syncthreads();
        if (tid < kBM) row_mask[tid] = (tid < nrows) ? p.pair_mask[p0 + tid] : 0ull;
        __syncthreads();
        if (tid < kBM / 16) {
            uint64_t m = 0;
            for (int r = 0; r < 16; ++r) m |= row_mask[tid * 16 + r];
            sub_mask[tid] = m;
        }
        __syncthreads();
        uint64_t tmask = 0, wsub[4];
#pragma unroll
        for (int i = 0; i < kBM / 16; ++i) tmask |= sub_mask[i];
#pragma unroll
        for (int i = 0; i < 4; ++i) wsub[i] = sub_mask[wm * 4 + i];
        const u16* W = p.Wdown + (size_t)e * p.d * p.H;
        f32x4 acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int c = 0; c < p.B; ++c) {
            if (!((tmask >> c) & 1ull)) continue;
            for (int kc = 0; kc < p.M; kc += kBK) {
                for (int i = tid; i < kBM * 8; i += kFfnThreads) {
                    const int r = i >> 3, ch = i & 7;
                    u32x4 v = {0u, 0u, 0u, 0u};
                    if ((row_mask[r] >> c) & 1ull)
                        v = ld16(p.Hbuf + (size_t)(p0 + r) * p.H + (size_t)c * p.M + kc + ch * 8);
                    st16(As + r * kLdk + ch * 8, v);
                }
                for (int i = tid; i < kBN * 8; i += kFfnThreads) {
                    const int r = i >> 3, ch = i & 7;
                    st16(Bs + r * kLdk + ch * 8,
                         ld16(W + (size_t)(n0 + r) * p.H + (size_t)c * p.M + kc + ch * 8));
                }
                __syncthreads();
#pragma unroll
                for (int kk = 0; kk < kBK; kk += 32) {
                    bf16x8 bw[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        bw[j] = as_bf16x8(ld16(Bs + (wn * 64 + j * 16 + frag_r) * kLdk + kk + frag_k));
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if ((wsub[i] >> c) & 1ull) {
                            const bf16x8 af =
                                as_bf16x8(ld16(As + (wm * 64 + i * 16 + frag_r) * kLdk + kk + frag_k));
#pragma unroll
                            for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(af, bw[j], acc[i][j]);
                        }
                    }
                }
                __syncthreads();
            }
        }
        // fp32 per-expert rows; each 16-lane group writes 64 contiguous bytes.
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = wm * 64 + i * 16 + (lane >> 4) * 4 + r;
                if (row < nrows) {
                    float* dst = p.part + (size_t)(p0 + row) * p.d + n0 + wn * 64 + (lane & 15);
#pragma unroll
                    for (int j = 0; j < 4; ++j) dst[j * 16] = acc[i][j][r];
                }
            }
    }
}

}  // namespace unifmoe
