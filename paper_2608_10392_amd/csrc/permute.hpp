// Token permutation and segment offsets.
//
// A "pair" is one (token, expert) evaluation: the shared expert on the
// token's blocks I_shr, or one of its k residual experts on I_res
// (Eq. selected-shared-output, selected-residual-output). Pairs are laid out
// grouped by expert and, inside an expert, by the Gray-code rank of the top
// key_bits bits of their block mask (a counting sort, see mask_key), so that
// pairs that share blocks sit next to each other for the down-projection
// tiles. Each (expert, block) "slab" gets the list of pairs that use it,
// which the up-projection tiles read.
//
//   route_kernel       counts pairs per (expert, key), taking each pair's slot
//                      in its bin, and rows per slab
//   scan_kernel        one workgroup per expert and one more: LDS-staged
//                      exclusive prefix sums -> bin cursors, expert segment
//                      offsets, slab offsets, chunk offsets, tile offsets
//   scatter_kernel     one thread per token writes its pairs at their slots
//   tables_kernel      down row tiles (per row tile), and per chunk of
//                      kChunk pairs of one expert: pairs per block
//   chunk_scan_kernel  per slab: exclusive scan of its chunk counts
//   slabfill_kernel    per chunk: each pair writes itself into the slabs of
//                      its blocks, in pair order (deterministic); per
//                      (expert, block group): the up tile table
//
// Each slab's row list starts at a multiple of the up-projection tile height
// bm_up and holds the slab's pairs in pair order, with their tokens beside
// them, so a tile's gather needs no dependent lookups. Up tiles are listed
// expert by expert, and inside an expert by groups of blocks, then by the
// stretch of the expert's pairs they cover (see up_tiles_of_group).
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kScanThreads = 1024;
constexpr int kChunk = 256;   // pairs per chunk of the ordered slab fill
constexpr int kXcdSlices = 8; // the down tile table is split into one slice per XCD

struct PermuteParams {
    int N, K, B, key_bits, bm_up, bm_down, down_col_tiles, up_group;
    const uint64_t* mask;
    const int* nres;
    const int* eids;
    const int* bin_count;
    int* bin_cursor;
    const int* slab_count;
    int* slab_off;
    int* seg_off;
    int* up_tile_off;
    int* down_tile_off;  // [K+2] first down row tile of each expert segment
    int* totals;  // [0] pairs P, [1] up tiles, [2] down tiles, [3] fill chunks, [4] down row tiles
    int* pair_token;
    uint64_t* pair_mask;
    int* pair_expert;
    int* pair_of;  // [N][K+1]: pair of the shared expert, then of q_1..q_k
    int* slab_rows;     // pair of each slab row (entries past a slab's count are unused)
    int* slab_tok;      // token of each slab row
    int* up_tile_info;  // per up tile: slab | rows << 16
    int* up_tile_rows;  // per up tile: first entry in slab_rows / slab_tok
    int* chunk_off;     // [K+2] first chunk of each expert's pair segment
    int* chunk_cnt;     // [chunks][B] pairs per block, then (scanned) first slab row
    int4* rt_info;      // per down row tile: first pair, rows, expert, cost (see down_rowtile)
    uint64_t* rt_masks; // per down row tile: mask union of each 16-row group, then of the tile
    int* down_tiles;    // per down tile: row tile << 8 | column tile
    int* down_slices;   // [9]: first down tile of each XCD's slice of the table, then the count
};

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

// Exclusive prefix sum of get(0..n-1) by one workgroup: each thread sums a
// contiguous chunk, the chunk sums are scanned in LDS, then each thread
// writes its chunk. Returns the total (same value in every thread).
template <class Get, class Put>
__device__ int block_exclusive_scan(int n, Get get, Put put, int* lds) {
    const int tid = threadIdx.x, T = blockDim.x;
    const int per = ceil_div(n, T);
    const int beg = min(n, tid * per), end = min(n, beg + per);
    int s = 0;
    for (int i = beg; i < end; ++i) s += get(i);
    lds[tid] = s;
    __syncthreads();
    for (int off = 1; off < T; off <<= 1) {
        const int v = (tid >= off) ? lds[tid - off] : 0;
        __syncthreads();
        lds[tid] += v;
        __syncthreads();
    }
    int run = lds[tid] - s;
    const int total = lds[T - 1];
    for (int i = beg; i < end; ++i) {
        const int c = get(i);
        put(i, run);
        run += c;
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
            for (int u = 0; u < 8; ++u) v[u] = (i0 + u * T < cnt) ? get(base + i0 + u * T) : 0;
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (i0 + u * T < cnt) stage[i0 + u * T] = v[u];
        }
        __syncthreads();
        const int per = ceil_div(cnt, T);
        const int beg = min(cnt, tid * per), end = min(cnt, beg + per);
        int s = 0;
        for (int i = beg; i < end; ++i) s += stage[i];
        lds[tid] = s;
        __syncthreads();
        for (int off = 1; off < T; off <<= 1) {
            const int v = (tid >= off) ? lds[tid - off] : 0;
            __syncthreads();
            lds[tid] += v;
            __syncthreads();
        }
        int run = carry + lds[tid] - s;
        const int total = lds[T - 1];
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

// One workgroup per expert, and one more. The routing kernel leaves the row
// counts per slab and the pair counts per expert in kSlabCopies copies
// (slab_count: [copy][nslab + K + 1]). Every workgroup sums the expert
// counts into the segment offsets; workgroup e <= K scans its expert's bins
// from its segment start; workgroup K + 1 builds the slab offsets and the
// tile offsets meanwhile.
__global__ __launch_bounds__(kScanThreads) void scan_kernel(PermuteParams p) {
    __shared__ int lds[kScanThreads];
    __shared__ int stage[kScanStage];
    __shared__ int segs[66];   // K + 2 <= 66
    const int K1 = p.K + 1, nslab = K1 * p.B, ncnt = nslab + K1, nb = 1 << p.key_bits;
    const int e = blockIdx.x;
    int* cnt = const_cast<int*>(p.slab_count);
    if ((int)threadIdx.x < K1) {
        int v[kSlabCopies];
#pragma unroll
        for (int c = 0; c < kSlabCopies; ++c) v[c] = cnt[(size_t)c * ncnt + nslab + threadIdx.x];
        int n = 0;
#pragma unroll
        for (int c = 0; c < kSlabCopies; ++c) n += v[c];
        lds[threadIdx.x] = n;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int x = 0; x < K1; ++x) {
            segs[x] = run;
            run += lds[x];
        }
        segs[K1] = run;
    }
    __syncthreads();
    if (e < K1) {
        const int base = segs[e];
        staged_exclusive_scan(
            nb, [&](int i) { return p.bin_count[(size_t)e * nb + i]; },
            [&](int i, int v) { p.bin_cursor[(size_t)e * nb + i] = base + v; }, stage, lds);
        return;
    }
    for (int x = threadIdx.x; x <= K1; x += blockDim.x) p.seg_off[x] = segs[x];
    const int P = segs[K1];
    // Row counts per slab: sum the copies into the first.
    for (int i = threadIdx.x; i < nslab; i += blockDim.x) {
        int v[kSlabCopies];
#pragma unroll
        for (int c = 0; c < kSlabCopies; ++c) v[c] = cnt[(size_t)c * ncnt + i];
        int n = 0;
#pragma unroll
        for (int c = 0; c < kSlabCopies; ++c) n += v[c];
        cnt[i] = n;
    }
    __syncthreads();
    const int bm = p.bm_up;
    const int nup = staged_exclusive_scan(
        nslab, [&](int i) { return ceil_div(p.slab_count[i], bm); },
        [&](int i, int v) {
            p.up_tile_off[i] = v;
            p.slab_off[i] = v * bm;
        },
        stage, lds);
    if (threadIdx.x == 0) {
        p.slab_off[nslab] = nup * bm;
        p.up_tile_off[nslab] = nup;
        if (p.chunk_off != nullptr) {
            int q = 0;
            for (int x = 0; x < K1; ++x) {
                p.chunk_off[x] = q;
                q += ceil_div(segs[x + 1] - segs[x], kChunk);
            }
            p.chunk_off[K1] = q;
            p.totals[3] = q;
        }
        int run = 0;
        for (int x = 0; x < K1; ++x) {
            p.down_tile_off[x] = run;
            run += ceil_div(segs[x + 1] - segs[x], p.bm_down);
        }
        p.down_tile_off[K1] = run;
        p.totals[0] = P;
        p.totals[1] = nup;
        p.totals[2] = run * p.down_col_tiles;
        p.totals[4] = run;
    }
}

// One thread per token writes its pairs at bin start + the slot the routing
// kernel took for each (stored in pair_of, overwritten here with the pair).
__global__ void scatter_kernel(PermuteParams p) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= p.N) return;
    const int k = p.nres[t];
    if (k == 0) return;  // padded token (valid tokens have k >= 1)
    const int B = p.B, kb = p.key_bits, K1 = p.K + 1;
    const uint64_t full = (B == 64) ? ~0ull : ((1ull << B) - 1ull);
    const uint64_t m = p.mask[t], rm = ~m & full;
    const int ks = mask_key(m, B, kb);
    const int kr = mask_key(rm, B, kb);
    int* of = p.pair_of + (size_t)t * K1;
    const int* eid = p.eids + (size_t)t * p.K;
    const int pr = p.bin_cursor[ks] + of[0];
    // Residual pairs in batches: every load of a batch (experts, slots, bin
    // cursors) is issued before its stores, which the compiler may not move
    // loads across.
    constexpr int kBatch = 8;
    for (int i0 = 0; i0 < k; i0 += kBatch) {
        int e[kBatch], q[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            e[u] = (i0 + u < k) ? eid[i0 + u] : 0;
            q[u] = (i0 + u < k) ? of[1 + i0 + u] : 0;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            if (i0 + u < k) q[u] += p.bin_cursor[(e[u] << kb) + kr];
        if (i0 == 0) {
            p.pair_token[pr] = t;
            p.pair_mask[pr] = m;
            p.pair_expert[pr] = 0;
            of[0] = pr;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (i0 + u < k) {
                p.pair_token[q[u]] = t;
                p.pair_mask[q[u]] = rm;
                p.pair_expert[q[u]] = e[u];
                of[1 + i0 + u] = q[u];
            }
        }
    }
}

// Up tile table, built once the slab rows of every chunk are known. Tiles
// are listed expert by expert; inside an expert the blocks are taken in
// groups of up_group, and inside a group tile j of block c is placed by the
// chunk q of the expert's pairs in which its first row falls, then by c,
// then by j. Tiles that run close together in this order gather the token
// rows of the same stretch of the expert's pairs, which a group's weight
// slabs share in L2. One workgroup per (expert, group); each thread takes a
// contiguous range of the expert's chunks. tile_lo(i, c) is the first tile
// of slab c whose first row is at or after chunk i's first slab row.
__device__ __forceinline__ void up_tiles_of_group(const PermuteParams& p, int grp, int* lds) {
    const int ngr = ceil_div(p.B, p.up_group);
    const int e = grp / ngr, g = grp - e * ngr;
    const int c0 = g * p.up_group, c1 = min(p.B, c0 + p.up_group);
    const int q0 = p.chunk_off[e], nq = p.chunk_off[e + 1] - q0;
    const int bm = p.bm_up, sl0 = e * p.B;
    auto tile_lo = [&](int i, int c) {
        const int sl = sl0 + c;
        const int r = (i < nq) ? p.chunk_cnt[(size_t)(q0 + i) * p.B + c] - p.slab_off[sl] : p.slab_count[sl];
        return ceil_div(r, bm);
    };
    const int tid = threadIdx.x, T = blockDim.x;
    const int per = ceil_div(nq, T);
    const int qa = min(nq, tid * per), qb = min(nq, qa + per);
    int n = 0;
    for (int c = c0; c < c1; ++c) n += tile_lo(qb, c) - tile_lo(qa, c);
    lds[tid] = n;
    __syncthreads();
    for (int off = 1; off < T; off <<= 1) {
        const int v = (tid >= off) ? lds[tid - off] : 0;
        __syncthreads();
        lds[tid] += v;
        __syncthreads();
    }
    int pos = p.up_tile_off[sl0 + c0] + lds[tid] - n;
    for (int i = qa; i < qb; ++i)
        for (int c = c0; c < c1; ++c) {
            const int sl = sl0 + c, cnt = p.slab_count[sl];
            for (int j = tile_lo(i, c), je = tile_lo(i + 1, c); j < je; ++j, ++pos) {
                p.up_tile_info[pos] = sl | (min(bm, cnt - j * bm) << 16);
                p.up_tile_rows[pos] = p.slab_off[sl] + j * bm;
            }
        }
    __syncthreads();
}

// Down row tiles: bm_down consecutive pairs of one expert segment. One wave
// per row tile records its first pair, row count and expert, and the union
// of the block masks of each 16-row group and of the whole tile. Down tiles
// (row tile x column tile of d) are listed row tile by row tile: the column
// tiles of one row tile run side by side on one XCD and read its H rows
// from HBM once.
__device__ __forceinline__ void down_rowtile(const PermuteParams& p, int rt) {
    const int e = upper_index(p.down_tile_off, p.K + 1, rt);
    const int p0 = p.seg_off[e] + (rt - p.down_tile_off[e]) * p.bm_down;
    const int nrows = min(p.bm_down, p.seg_off[e + 1] - p0);
    const int lane = threadIdx.x & 63, G = p.bm_down / 16;
    uint64_t* out = p.rt_masks + (size_t)rt * (G + 1);
    uint64_t all = 0;
    int groups = 0;   // blocks summed over the 32-row MFMA groups (lanes 0 and 32)
    for (int h = 0; h * 64 < p.bm_down; ++h) {
        const int r = h * 64 + lane;
        uint64_t m = r < nrows ? p.pair_mask[p0 + r] : 0ull;
        for (int o = 1; o < 16; o <<= 1) m |= shfl_xor64(m, o);
        if ((lane & 15) == 0) out[h * 4 + (lane >> 4)] = m;
        all |= m;
        const uint64_t m32 = m | shfl_xor64(m, 16);
        if ((lane & 31) == 0) groups += __popcll(m32);
    }
    for (int o = 16; o < 64; o <<= 1) all |= shfl_xor64(all, o);
    groups += __shfl_xor(groups, 32);
    if (lane == 0) {
        out[G] = all;
        // Cost estimate for balancing the XCD slices: the MFMA work (blocks
        // over the 32-row groups) plus a per-stage share for the copies
        // every stage of the tile's union makes.
        p.rt_info[rt] = make_int4(p0, nrows, e, groups + 4 * __popcll(all));
    }
    for (int ct = lane; ct < p.down_col_tiles; ct += 64)
        p.down_tiles[(size_t)rt * p.down_col_tiles + ct] = (rt << 8) | ct;
}



// Chunk q of expert e covers pairs [seg_off[e] + (q - chunk_off[e]) kChunk, ...)
// of the expert's segment. One workgroup of kChunk threads per chunk, one
// thread per pair; workgroups past the chunk count exit.
struct ChunkView {
    int e, lo, hi;
};
__device__ __forceinline__ ChunkView chunk_view(const PermuteParams& p, int q) {
    ChunkView v;
    v.e = upper_index(p.chunk_off, p.K + 1, q);
    v.lo = p.seg_off[v.e] + (q - p.chunk_off[v.e]) * kChunk;
    v.hi = min(v.lo + kChunk, p.seg_off[v.e + 1]);
    return v;
}

// Pairs of the workgroup's waves that use each block (wave ballots).
__device__ __forceinline__ void chunk_wave_counts(int B, uint64_t m, int (*wc)[64]) {
    const int w = threadIdx.x >> 6;
    for (int c = 0; c < B; ++c) {
        const uint64_t bits = ballot(((m >> c) & 1ull) != 0ull);
        if (lane_id() == 0) wc[w][c] = __popcll(bits);
    }
}

// The two tables that only need the scatter's output, in one launch (each
// is small; a kernel launch costs more than their work): workgroups [0, g1)
// build the down row tiles (one wave per row tile), the rest count the
// chunks' rows per block.
__global__ __launch_bounds__(256) void tables_kernel(PermuteParams p, int g1) {
    static_assert(kChunk == 256, "one thread per chunk pair");
    __shared__ int wc[kChunk / 64][64];
    const int b = blockIdx.x;
    if (b < g1) {
        const int nrt = p.totals[4];
        for (int rt = b * 4 + (threadIdx.x >> 6); rt < nrt; rt += g1 * 4) down_rowtile(p, rt);
    } else {
        const int g2 = gridDim.x - g1, nq = p.totals[3];
        for (int q = b - g1; q < nq; q += g2) {
            const ChunkView v = chunk_view(p, q);
            const int pr = v.lo + (int)threadIdx.x;
            chunk_wave_counts(p.B, pr < v.hi ? p.pair_mask[pr] : 0ull, wc);
            __syncthreads();
            if ((int)threadIdx.x < p.B) {
                int n = 0;
                for (int w = 0; w < kChunk / 64; ++w) n += wc[w][threadIdx.x];
                p.chunk_cnt[(size_t)q * p.B + threadIdx.x] = n;
            }
            __syncthreads();
        }
    }
}

// The down tile table is split into one contiguous slice per XCD with equal
// estimated cost (rt_info[].w per tile of a row tile), not equal tile
// counts: the shared expert's row tiles, listed first, are cheaper. Slice x
// starts at the first tile whose preceding cost reaches x/8 of the total.
__device__ __forceinline__ void down_slices(const PermuteParams& p, int* lds) {
    const int nrt = p.totals[4], ncol = p.down_col_tiles;
    const int total = block_exclusive_scan(
        nrt, [&](int i) { return p.rt_info[i].w * ncol; }, [&](int, int) {}, lds);
    if (threadIdx.x == 0) {
        p.down_slices[0] = 0;
        p.down_slices[kXcdSlices] = nrt * ncol;
        for (int x = 1; x < kXcdSlices; ++x)
            if ((int64_t)x * total / kXcdSlices == 0) p.down_slices[x] = 0;
    }
    block_exclusive_scan(
        nrt, [&](int i) { return p.rt_info[i].w * ncol; },
        [&](int i, int v) {
            const int c = p.rt_info[i].w;
            for (int x = 1; x < kXcdSlices; ++x) {
                const int target = (int)((int64_t)x * total / kXcdSlices);
                if (target > v && target <= v + ncol * c)
                    p.down_slices[x] = i * ncol + (target - v + c - 1) / c;
            }
        },
        lds);
}

// One workgroup per slab: its chunks' counts become the slab row at which
// each chunk's pairs start. One more workgroup splits the down tile table
// into the XCD slices.
__global__ __launch_bounds__(256) void chunk_scan_kernel(PermuteParams p) {
    __shared__ int lds[256];
    if ((int)blockIdx.x == (p.K + 1) * p.B) {
        down_slices(p, lds);
        return;
    }
    const int sl = blockIdx.x;
    const int e = sl / p.B, c = sl - e * p.B;
    const int q0 = p.chunk_off[e], nq = p.chunk_off[e + 1] - q0;
    const int base = p.slab_off[sl];
    int* cnt = p.chunk_cnt + (size_t)q0 * p.B + c;
    block_exclusive_scan(
        nq, [&](int i) { return cnt[(size_t)i * p.B]; }, [&](int i, int v) { cnt[(size_t)i * p.B] = base + v; },
        lds);
}

// first[c]: the chunk's first row in slab c, staged in LDS so that the
// store loop below carries no global loads.
__device__ __forceinline__ void slabfill_chunk(const PermuteParams& p, int q, int (*wc)[64], int* first) {
    const ChunkView v = chunk_view(p, q);
    const int pr = v.lo + (int)threadIdx.x;
    const bool act = pr < v.hi;
    const uint64_t m = act ? p.pair_mask[pr] : 0ull;
    const int tok = act ? p.pair_token[pr] : 0;
    if ((int)threadIdx.x < p.B) first[threadIdx.x] = p.chunk_cnt[(size_t)q * p.B + threadIdx.x];
    chunk_wave_counts(p.B, m, wc);
    __syncthreads();
    const int w = threadIdx.x >> 6;
    for (int c = 0; c < p.B; ++c) {
        const bool use = ((m >> c) & 1ull) != 0ull;
        const uint64_t bits = ballot(use);
        if (use) {
            int at = first[c] + __popcll(bits & lanes_below());
            for (int w2 = 0; w2 < w; ++w2) at += wc[w2][c];
            p.slab_rows[at] = pr;
            p.slab_tok[at] = tok;
        }
    }
}

// Workgroups [0, n_groups) build the up tile table of one (expert, block
// group) each; the rest fill the chunks' slab rows.
__global__ __launch_bounds__(kChunk) void slabfill_kernel(PermuteParams p, int n_groups) {
    __shared__ int wc[kChunk / 64][64];
    __shared__ int first[64];
    const int b = blockIdx.x;
    if (b < n_groups) {
        up_tiles_of_group(p, b, &wc[0][0]);
        return;
    }
    const int nq = p.totals[3];
    for (int q = b - n_groups; q < nq; q += gridDim.x - n_groups) {
        slabfill_chunk(p, q, wc, first);
        __syncthreads();
    }
}

}  // namespace unifmoe
