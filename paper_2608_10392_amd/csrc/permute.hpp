// Token permutation and segment offsets.
//
// A "pair" is one (token, expert) evaluation: the shared expert on the
// token's blocks I_shr, or one of its k residual experts on I_res
// (Eq. selected-shared-output, selected-residual-output). Pairs are laid out
// grouped by expert and, inside an expert, by the Gray-code rank of the top
// key_bits bits of their block mask (a counting sort, see mask_key), so that
// pairs that share blocks sit next to each other for the down-projection
// tiles. Each (expert, block) "slab" gets the list of pairs that use it, in
// token order, which the up-projection tiles read (and the backward's weight
// gradients sum over, in that order).
//
//   route kernels  per pair, its slot in its (expert, key) bin copy; per
//                  tile of 64 tokens, rows per slab and pairs per expert
//                  (tile_cnt), and the pairs per expert
//   scan_kernel    one workgroup per expert: pairs per expert, segments,
//                  bin cursors; one per slab: the exclusive prefix of its
//                  rows over the token tiles, and its total
//   scatter_kernel one workgroup per token tile: pairs at their slots, and
//                  every slab row (the tile's first row in the slab plus the
//                  token's rank among the tile's tokens that use the slab,
//                  from a ballot); one workgroup per (expert, block group):
//                  the up tile table
//
// Each slab's row list starts at a multiple of the up-projection tile height
// bm_up and holds the slab's pairs with their tokens beside them, so a
// tile's gather needs no dependent lookups. Up tiles are listed expert by
// expert, and inside an expert by groups of blocks, then by the token tile
// in which they start (see up_tiles_of_group). Down tiles are described by
// the down kernel itself from the expert segments.
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kScanThreads = 1024;
constexpr int kPermTok = 64;     // tokens per tile of the counts and the scatter (one wave)

struct PermuteParams {
    int N, K, B, key_bits, bm_up, bm_down, down_col_tiles, up_group, ntile;
    int max_pairs;      // pairs the pair-indexed buffers hold (the workspace's capacity)
    const uint64_t* mask;
    const int* nres;
    const int* eids;
    const int* bin_count;   // [kBinCopies][(K+1) << key_bits] (bin_counter)
    int* bin_cursor;        // [(K+1) << key_bits][kBinCopies]
    int* slab_count;    // [nslab] rows per slab (the scan's column sums)
    int* slab_off;      // [nslab + 1] first entry of each slab in the row lists (bf16)
    int* tile_cnt;      // [ntile][nslab + K + 1] per-tile counts; the scan turns each slab column into
                        // the tile's first row in the slab (exclusive prefix over tiles)
    const int* exp_total;   // [kExpCopies][K + 1] pairs per expert
    const int* pair_rank;   // [N][K + 1] slot of each pair within its bin copy
    int* seg_off;
    int* down_tile_off;  // [K+2] first down row tile of each expert segment
    int* totals;  // [0] pairs P, [1] up tiles, [2] down tiles, [4] down row tiles, [5] P > max_pairs
    int* pair_token;
    uint64_t* pair_mask;
    int* pair_expert;
    int* pair_of;  // [N][K+1]: the pairs of the shared expert and of q_1..q_k
    int* slab_rows;     // pair of each slab row (entries past a slab's count are unused)
    int* slab_tok;      // token of each slab row
    int* up_tile_info;  // per up tile: slab | rows << 16
    int* up_tile_rows;  // per up tile: first entry in slab_rows / slab_tok
    int4* rt_info;      // per down row tile: first pair, rows, expert, blocks in its union
    uint64_t* rt_masks; // per down row tile: mask union of each 32-row group, then of the tile
    int* down_slices;   // [kXcds + 1]: the down tiles each XCD's queue owns (down_tables)
    int down_stages;    // stages per block of the down-projection (M / 64)
    int down_splits;    // parts each down row tile is split into (DownParams::nsplit)
};

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

// Exclusive prefix over the workgroup (thread order) of each thread's s, and
// the total in every thread: an inclusive scan inside each wave with
// shuffles, then the wave totals through lds (at least blockDim.x / 64
// words). Two barriers instead of two per doubling step; lds is free again
// on return. blockDim.x is a multiple of 64, at most 1024.
__device__ __forceinline__ int block_prefix(int s, int* lds, int& total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int x = s;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) lds[w] = x;
    __syncthreads();
    int base = 0, tot = 0;
    for (int i = 0; i < nw; ++i) {
        const int v = lds[i];
        base += (i < w) ? v : 0;
        tot += v;
    }
    __syncthreads();
    total = tot;
    return base + x - s;
}

// Exclusive prefix sum of get(0..n-1) by one workgroup: each thread sums a
// contiguous chunk, the chunk sums are scanned in LDS, then each thread
// writes its chunk. Returns the total (same value in every thread).
template <class Get, class Put>
__device__ int block_exclusive_scan(int n, Get get, Put put, int* lds) {
    const int tid = threadIdx.x, T = blockDim.x;
    const int per = ceil_div(n, T);
    const int beg = min(n, tid * per), end = min(n, beg + per);
    // Up to 8 values per thread are loaded together into registers (their
    // latencies overlap), longer chunks are read twice.
    constexpr int R = 8;
    int v[R];
    if (per <= R && n > 0) {
        // Every load is issued (past the chunk: the last element again, then
        // dropped), so none waits behind a branch for the previous one.
#pragma unroll
        for (int u = 0; u < R; ++u) {
            const int x = get(min(beg + u, n - 1));
            v[u] = (beg + u < end) ? x : 0;
        }
    } else if (per <= R) {
#pragma unroll
        for (int u = 0; u < R; ++u) v[u] = 0;
    }
    int s = 0;
    if (per <= R) {
#pragma unroll
        for (int u = 0; u < R; ++u) s += v[u];
    } else {
        for (int i = beg; i < end; ++i) s += get(i);
    }
    int total;
    int run = block_prefix(s, lds, total);
    if (per <= R) {
#pragma unroll
        for (int u = 0; u < R; ++u)
            if (beg + u < end) {
                put(beg + u, run);
                run += v[u];
            }
    } else {
        for (int i = beg; i < end; ++i) {
            const int c = get(i);
            put(i, run);
            run += c;
        }
    }
    __syncthreads();
    return total;
}

// The same for long inputs: pieces of up to kScanStage values are loaded
// into LDS with consecutive (coalesced, independent) reads, scanned there,
// and written back the same way, so the global latency is paid a few times
// per piece instead of once per value of a thread's chunk.
constexpr int kScanStage = 16384;
template <class Get, class Put>
__device__ int staged_exclusive_scan(int n, Get get, Put put, int* stage, int* lds) {
    const int tid = threadIdx.x, T = blockDim.x;
    int carry = 0;
    for (int base = 0; base < n; base += kScanStage) {
        const int cnt = min(kScanStage, n - base);
        // Loads in batches of 8 per thread, all issued before any is stored.
        for (int i0 = tid; i0 < cnt; i0 += 8 * T) {
            int v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = get(base + min(i0 + u * T, cnt - 1));
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (i0 + u * T < cnt) stage[i0 + u * T] = v[u];
        }
        __syncthreads();
        const int per = ceil_div(cnt, T);
        const int beg = min(cnt, tid * per), end = min(cnt, beg + per);
        int s = 0;
        for (int i = beg; i < end; ++i) s += stage[i];
        int total;
        int run = carry + block_prefix(s, lds, total);
        for (int i = beg; i < end; ++i) {
            const int c = stage[i];
            stage[i] = run;
            run += c;
        }
        __syncthreads();
        for (int i = tid; i < cnt; i += T) put(base + i, stage[i]);
        carry += total;
        __syncthreads();
    }
    return carry;
}

// Workgroups [0, K]: expert segments (from the routing tiles' pair totals),
// then expert e's bin cursors (its segment start plus the
// exclusive prefix of its bins); workgroup 0 also writes the segments, the
// down row-tile offsets and the totals. Workgroups past them: slab
// sl = blockIdx.x - K - 1, its rows per token tile turned into each tile's
// first row in the slab, and its total.
__global__ __launch_bounds__(kScanThreads) void scan_kernel(PermuteParams p) {
    __shared__ int lds[kScanThreads];
    __shared__ int stage[kScanStage];
    __shared__ int segs[66];   // K + 2 <= 66
    const int K1 = p.K + 1, nslab = K1 * p.B, ncnt = nslab + K1, nb = 1 << p.key_bits;
    const int b = blockIdx.x;
    const int tid = threadIdx.x, T = blockDim.x;
    if (b >= K1) {
        const int sl = b - K1;
        const int total = block_exclusive_scan(
            p.ntile, [&](int i) { return p.tile_cnt[(size_t)i * ncnt + sl]; },
            [&](int i, int v) { p.tile_cnt[(size_t)i * ncnt + sl] = v; }, lds);
        if (tid == 0) p.slab_count[sl] = total;
        return;
    }
    // Pairs per expert: the routing tiles' totals.
    if (tid < K1) {
        int n = 0;
#pragma unroll
        for (int c = 0; c < kExpCopies; ++c) n += p.exp_total[c * K1 + tid];
        segs[tid] = n;
    }
    __syncthreads();
    if (tid == 0) {
        int run = 0;
        for (int x = 0; x < K1; ++x) {
            const int n = segs[x];
            segs[x] = run;
            run += n;
        }
        segs[K1] = run;
    }
    __syncthreads();
    if (b == 0) {
        for (int x = tid; x <= K1; x += T) p.seg_off[x] = segs[x];
        if (tid == 0) {
            int run = 0;
            for (int x = 0; x < K1; ++x) {
                p.down_tile_off[x] = run;
                run += ceil_div(segs[x + 1] - segs[x], p.bm_down);
            }
            p.down_tile_off[K1] = run;
            // More pairs than the buffers hold: no down tiles, and the flag
            // that makes the scatter, the fp32 FFN and the merge stand down
            // (the up tile count stays at its cleared 0).
            const bool over = segs[K1] > p.max_pairs;
            p.totals[0] = segs[K1];
            p.totals[2] = over ? 0 : run * p.down_col_tiles;
            p.totals[4] = over ? 0 : run;
            p.totals[5] = over ? 1 : 0;
        }
    }
    // Expert b's bins in key order, each bin's copies in copy order; the
    // cursors keep this order (a bin's kBinCopies cursors are consecutive).
    const int base = segs[b], nbin = K1 * nb;
    const size_t off = (size_t)b * nb * kBinCopies;
    staged_exclusive_scan(
        nb * kBinCopies,
        [&](int i) { return p.bin_count[bin_counter(b * nb + i / kBinCopies, i % kBinCopies, nbin)]; },
        [&](int i, int v) { p.bin_cursor[off + i] = base + v; }, stage, lds);
}

// Slab offsets, in LDS (each scatter workgroup computes them): slab sl
// starts at so[sl] (a multiple of bm_up) and its up tiles at uo[sl]
// (so[nslab], uo[nslab]: the totals). Workgroup 0 records the up tile count.
__device__ __forceinline__ void slab_offsets(const PermuteParams& p, int* so, int* uo, int* lds) {
    const int nslab = (p.K + 1) * p.B, bm = p.bm_up;
    const int nup = block_exclusive_scan(
        nslab, [&](int i) { return ceil_div(p.slab_count[i], bm); },
        [&](int i, int v) {
            uo[i] = v;
            so[i] = v * bm;
        },
        lds);
    if (threadIdx.x == 0) {
        uo[nslab] = nup;
        so[nslab] = nup * bm;
        if (blockIdx.x == 0) p.totals[1] = nup;
    }
    __syncthreads();
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i <= nslab; i += blockDim.x) p.slab_off[i] = so[i];
}

// Up tile table. Tiles are listed expert by expert; inside an expert the
// blocks are taken in groups of up_group, and inside a group tile j of block
// c is placed by the chunk of token tiles in which its first row falls, then
// by c, then by j. Tiles that run close together in this order gather the
// token rows of the same stretch of tokens, which a group's weight slabs
// share in L2. One workgroup per (expert, group). A chunk is CH token tiles,
// CH chosen so that the group's first up tile of every chunk,
// tl[i][c] = ceil(first row of chunk i in slab c / bm_up), fits in
// kUpTableWords words of LDS; these are loaded first (coalesced), then each
// thread takes a contiguous range of chunks.
constexpr int kUpTableWords = 8192;
__device__ __forceinline__ void up_tiles_of_group(const PermuteParams& p, int grp, const int* so, const int* uo,
                                                  int* lds) {
    const int ngr = ceil_div(p.B, p.up_group);
    const int e = grp / ngr, g = grp - e * ngr;
    const int c0 = g * p.up_group, c1 = min(p.B, c0 + p.up_group), ng = c1 - c0;
    const int ncnt = (p.K + 1) * (p.B + 1);
    const int bm = p.bm_up, sl0 = e * p.B;
    // (nq + 1) ng <= (ntile / CH + 2) ng < kUpTableWords, since ng <= 64)
    const int CH = max(1, ceil_div((p.ntile + 1) * ng, kUpTableWords - 256));
    const int nq = ceil_div(p.ntile, CH);
    int* tl = lds;                           // [nq + 1][ng]
    int* scan = lds + kUpTableWords;         // blockDim.x words
    int* cn = scan + blockDim.x;             // [ng] rows of the group's slabs
    batched_copy(
        (nq + 1) * ng,
        [&](int x) {
            const int i = x / ng, sl = sl0 + c0 + x - i * ng;
            return (i < nq) ? p.tile_cnt[(size_t)i * CH * ncnt + sl] : p.slab_count[sl];
        },
        [&](int x, int r) {
            tl[x] = ceil_div(r, bm);
            if (x >= nq * ng) cn[x - nq * ng] = r;
        });
    __syncthreads();
    const int tid = threadIdx.x, T = blockDim.x;
    const int per = ceil_div(nq, T);
    const int qa = min(nq, tid * per), qb = min(nq, qa + per);
    int n = 0;
    for (int c = 0; c < ng; ++c) n += tl[qb * ng + c] - tl[qa * ng + c];
    int ntot;
    int pos = uo[sl0 + c0] + block_prefix(n, scan, ntot);
    for (int i = qa; i < qb; ++i)
        for (int c = 0; c < ng; ++c) {
            const int sl = sl0 + c0 + c, cnt = cn[c], s0 = so[sl];
            for (int j = tl[i * ng + c], je = tl[(i + 1) * ng + c]; j < je; ++j, ++pos) {
                p.up_tile_info[pos] = sl | (min(bm, cnt - j * bm) << 16);
                p.up_tile_rows[pos] = s0 + j * bm;
            }
        }
    __syncthreads();
}

// One workgroup of kScatterWaves waves per token tile (lane = token). Each
// pair goes to its bin copy's cursor plus the slot the routing kernel took.
// Wave w takes the residual pairs i = w, w + kScatterWaves, .. of the tile's
// tokens (wave 0 also the shared pairs). Then, slab by slab, the tile's
// tokens that use the slab take consecutive rows from the tile's first row
// in it, in token order (ballot ranks), so every slab lists its tokens in
// token order; wave w takes experts w, w + kScatterWaves, .. The tokens'
// pairs per expert and the tile's first rows are staged in LDS.
constexpr int kScatterWaves = 4;
__device__ __forceinline__ void scatter_tile(const PermuteParams& p, int q, const int* so, int* pidx, int* first) {
    const int lane = lane_id(), t = q * kPermTok + lane;
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int K = p.K, K1 = K + 1, B = p.B, kb = p.key_bits, nslab = K1 * B;
    const int ncnt = nslab + K1;
    const bool in = t < p.N;
    const int k = in ? p.nres[t] : 0;   // 0 for padded tokens (valid tokens have k >= 1)
    const bool v = k > 0;
    const uint64_t full = (B == 64) ? ~0ull : ((1ull << B) - 1ull);
    const uint64_t m = v ? p.mask[t] : 0ull, rm = ~m & full;
    int* of = p.pair_of + (size_t)(v ? t : 0) * K1;
    const int* eid = p.eids + (size_t)(v ? t : 0) * K;
    const bool slabs = p.slab_rows != nullptr;   // no slab lists for fp32 layers
    // The tile's first row in each slab (absolute), read while the pairs'
    // atomics are in flight.
    const int* tfirst = p.tile_cnt + (size_t)q * ncnt;
    if (slabs)
        batched_copy(nslab, [&](int sl) { return tfirst[sl]; }, [&](int sl, int v) { first[sl] = so[sl] + v; });
    uint64_t sel = 0;
    const int bc = q % kBinCopies;   // the bin copy of this token tile
    if (v) {
        const int kr = mask_key(rm, B, kb);
        // This wave's residual pairs, in batches: every load of a batch is
        // issued before its results are used.
        constexpr int kBatch = 4;
        const int* rank = p.pair_rank + (size_t)t * K1;
        for (int i0 = wave; i0 < k; i0 += kBatch * kScatterWaves) {
            int e[kBatch], r[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int i = i0 + u * kScatterWaves;
                e[u] = (i < k) ? eid[i] : 0;
                r[u] = (i < k) ? rank[1 + i] : 0;
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u)
                if (i0 + u * kScatterWaves < k) r[u] += p.bin_cursor[((e[u] << kb) + kr) * kBinCopies + bc];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int i = i0 + u * kScatterWaves;
                if (i < k) {
                    p.pair_token[r[u]] = t;
                    p.pair_mask[r[u]] = rm;
                    p.pair_expert[r[u]] = e[u];
                    of[1 + i] = r[u];
                    pidx[lane * K1 + e[u]] = r[u];
                }
            }
        }
        if (wave == 0) {
            const int pr = p.bin_cursor[mask_key(m, B, kb) * kBinCopies + bc] + p.pair_rank[(size_t)t * K1];
            p.pair_token[pr] = t;
            p.pair_mask[pr] = m;
            p.pair_expert[pr] = 0;
            of[0] = pr;
            pidx[lane * K1] = pr;
        }
        for (int i = 0; i < k; ++i) sel |= 1ull << (eid[i] - 1);
    }
    if (!slabs) return;
    __syncthreads();
    // Slab rows of this wave's experts (an expert none of the tile's tokens
    // uses is skipped whole).
    const uint64_t below = lanes_below();
    for (int e = wave; e <= K; e += kScatterWaves) {
        const bool he = (e == 0) ? v : ((sel >> (e - 1)) & 1ull) != 0ull;
        if (!ballot(he)) continue;
        const uint64_t me = (e == 0) ? m : rm;
        const int pr = he ? pidx[lane * K1 + e] : 0;
        // The expert's first rows, one slab per lane (B <= 64), read back
        // per slab from a register instead of LDS.
        const int fe = (lane < B) ? first[e * B + lane] : 0;
        for (int c = 0; c < B; ++c) {
            const bool has = he && ((me >> c) & 1ull);
            const uint64_t bits = ballot(has);
            if (!bits) continue;
            if (has) {
                const int at = __builtin_amdgcn_readlane(fe, c) + __popcll(bits & below);
                p.slab_rows[at] = pr;
                p.slab_tok[at] = t;
            }
        }
    }
}

// Workgroups [0, n_groups) build the up tile table of one (expert, block
// group) each; the rest scatter one token tile each.
__global__ __launch_bounds__(kScatterWaves * 64) void scatter_kernel(PermuteParams p, int n_groups) {
    // Routing needed more pairs than the buffers hold: nothing to place.
    if (ld_uniform(p.totals + 5) != 0) return;
    // LDS: slab and up tile offsets ([nslab + 1] each), then the role's
    // words: the tokens' pairs [64][K+1] and the tile's first rows [nslab],
    // or the up table's inputs.
    extern __shared__ int lds_sc[];
    const int nslab = (p.K + 1) * p.B;
    int* so = lds_sc;
    int* uo = so + nslab + 1;
    int* rest = uo + nslab + 1;
    if (p.slab_rows != nullptr) slab_offsets(p, so, uo, rest);
    const int b = blockIdx.x;
    if (b < n_groups) {
        up_tiles_of_group(p, b, so, uo, rest);
        return;
    }
    scatter_tile(p, b - n_groups, so, rest, rest + 64 * (p.K + 1));
}

// Down row tiles: bm_down consecutive pairs of one expert segment. One wave
// per row tile records its first pair, row count and expert, and the union
// of the block masks of each 32-row group and of the whole tile (the down
// kernel contracts over the tile's union and skips, per 32-row MFMA group,
// the blocks none of its rows use).
__global__ __launch_bounds__(256) void down_tables_kernel(PermuteParams p) {
    const int nrt = p.totals[4], G = p.bm_down / 32;
    const int lane = lane_id();
    for (int rt = blockIdx.x * 4 + ((int)threadIdx.x >> 6); rt < nrt; rt += gridDim.x * 4) {
        const int e = upper_index(p.down_tile_off, p.K + 1, rt);
        const int p0 = p.seg_off[e] + (rt - p.down_tile_off[e]) * p.bm_down;
        const int nrows = min(p.bm_down, p.seg_off[e + 1] - p0);
        uint64_t* out = p.rt_masks + (size_t)rt * (G + 1);
        uint64_t m[4];   // bm_down <= 256: rows h * 64 + lane
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            const int r = h * 64 + lane;
            m[h] = (h * 64 < p.bm_down && r < nrows) ? p.pair_mask[p0 + r] : 0ull;
        }
        uint64_t all = 0;
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            uint64_t g = m[h];
#pragma unroll
            for (int o = 1; o < 32; o <<= 1) g |= shfl_xor64(g, o);
            if ((lane & 31) == 0 && h * 64 < p.bm_down) out[h * 2 + (lane >> 5)] = g;
            all |= g;
        }
        all |= shfl_xor64(all, 32);
        if (lane == 0) {
            out[G] = all;
            p.rt_info[rt] = make_int4(p0, nrows, e, __popcll(all));
        }
    }
}

// The down tiles split over the XCDs' queues by cost instead of by count
// (one workgroup, after down_tables): a row tile's tiles cost about its
// stages (at least 4) plus 2 for each tile's epilogue and hand-over, per
// column tile and part. XCD x takes the row tiles from the first whose
// exclusive cost prefix reaches x / kXcds of the total: r + 1 for the one
// row tile r whose cost interval (prefix(r), prefix(r) + cost(r)] holds that
// target (costs are positive, so the intervals tile (0, total] and the
// boundaries never decrease), 0 for a target of 0.
constexpr int kSliceThreads = 1024;
__global__ __launch_bounds__(kSliceThreads) void down_slices_kernel(PermuteParams p) {
    __shared__ int part[kSliceThreads / 64];
    __shared__ int bound[kXcds + 1];
    const int nrt = p.totals[4], ns = p.down_splits;
    const int T = blockDim.x, tid = threadIdx.x;
    const int per = ceil_div(nrt, T), r0 = min(nrt, tid * per), r1 = min(nrt, r0 + per);
    auto cost = [&](int rt) { return p.down_col_tiles * (max(p.rt_info[rt].w * p.down_stages, 4) + 2 * ns); };
    int sum = 0;
    for (int r = r0; r < r1; ++r) sum += cost(r);
    if (tid <= kXcds) bound[tid] = (tid == kXcds) ? nrt : 0;
    int itotal;
    long long run = block_prefix(sum, part, itotal);
    const long long total = itotal;
    for (int r = r0; r < r1; ++r) {
        const int c = cost(r);
        for (int x = 1; x < kXcds; ++x) {
            const long long target = total * x / kXcds;
            if (run < target && run + c >= target) bound[x] = r + 1;
        }
        run += c;
    }
    __syncthreads();
    if (tid <= kXcds) p.down_slices[tid] = bound[tid] * p.down_col_tiles * ns;
}

}  // namespace unifmoe
