// Token permutation and segment offsets.
//
// A "pair" is one (token, expert) evaluation: the shared expert on the
// token's blocks I_shr, or one of its k residual experts on I_res
// (Eq. selected-shared-output, selected-residual-output). Pairs are laid out
// grouped by expert and, inside an expert, by the top key_bits bits of their
// block mask (a counting sort), so that pairs that share blocks sit next to
// each other for the down-projection tiles. Each (expert, block) "slab" gets
// the list of pairs that use it, which the up-projection tiles read.
//
//   route_kernel   counts pairs per (expert, key) and rows per slab
//   scan_kernel    one workgroup: LDS-staged exclusive prefix sums -> bin
//                  cursors, expert segment offsets, slab offsets, tile tables
//   scatter_kernel one thread per token claims its pair slots
//   slabfill_kernel one thread per pair; wave ballots reserve slab slots
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kScanThreads = 1024;

struct PermuteParams {
    int N, K, B, key_bits, bm_up, bm_down, down_col_tiles;
    const uint64_t* mask;
    const int* nres;
    const int* eids;
    const int* bin_count;
    int* bin_cursor;
    const int* slab_count;
    int* slab_off;
    int* slab_cursor;
    int* seg_off;
    int* up_tile_off;
    int* down_tile_off;
    int* totals;  // [0] pairs P, [1] up-projection tiles, [2] down-projection tiles
    int* pair_token;
    uint64_t* pair_mask;
    int* pair_expert;
    int* pair_of;  // [N][K+1]: pair of the shared expert, then of q_1..q_k
    int* slab_rows;
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

__global__ __launch_bounds__(kScanThreads) void scan_kernel(PermuteParams p) {
    __shared__ int lds[kScanThreads];
    const int K1 = p.K + 1, nbin = K1 << p.key_bits, nslab = K1 * p.B;
    const int P = block_exclusive_scan(
        nbin, [&](int i) { return p.bin_count[i]; }, [&](int i, int v) { p.bin_cursor[i] = v; }, lds);
    for (int e = threadIdx.x; e <= K1; e += blockDim.x)
        p.seg_off[e] = (e < K1) ? p.bin_cursor[e << p.key_bits] : P;
    const int rows = block_exclusive_scan(
        nslab, [&](int i) { return p.slab_count[i]; },
        [&](int i, int v) { p.slab_off[i] = v; p.slab_cursor[i] = v; }, lds);
    const int bm = p.bm_up;
    const int nup = block_exclusive_scan(
        nslab, [&](int i) { return ceil_div(p.slab_count[i], bm); },
        [&](int i, int v) { p.up_tile_off[i] = v; }, lds);
    if (threadIdx.x == 0) {
        p.slab_off[nslab] = rows;
        p.up_tile_off[nslab] = nup;
        int run = 0;
        for (int e = 0; e < K1; ++e) {
            p.down_tile_off[e] = run;
            run += ceil_div(p.seg_off[e + 1] - p.seg_off[e], p.bm_down) * p.down_col_tiles;
        }
        p.down_tile_off[K1] = run;
        p.totals[0] = P;
        p.totals[1] = nup;
        p.totals[2] = run;
    }
}

__global__ void scatter_kernel(PermuteParams p) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= p.N) return;
    const int k = p.nres[t];
    if (k == 0) return;  // padded token (valid tokens have k >= 1)
    const int B = p.B, kb = p.key_bits, K1 = p.K + 1;
    const uint64_t full = (B == 64) ? ~0ull : ((1ull << B) - 1ull);
    const uint64_t m = p.mask[t], rm = ~m & full;
    const int ks = (int)(B > kb ? (m >> (B - kb)) : m);
    const int kr = (int)(B > kb ? (rm >> (B - kb)) : rm);
    int pr = atomicAdd(&p.bin_cursor[ks], 1);
    p.pair_token[pr] = t;
    p.pair_mask[pr] = m;
    p.pair_expert[pr] = 0;
    p.pair_of[(size_t)t * K1] = pr;
    for (int i = 0; i < k; ++i) {
        const int e = p.eids[(size_t)t * p.K + i];
        pr = atomicAdd(&p.bin_cursor[(e << kb) + kr], 1);
        p.pair_token[pr] = t;
        p.pair_mask[pr] = rm;
        p.pair_expert[pr] = e;
        p.pair_of[(size_t)t * K1 + 1 + i] = pr;
    }
}

// Persistent over pairs. Lanes of a wave hold consecutive pairs, which mostly
// share an expert; for each expert present and each block, one atomic
// reserves the slots of all lanes that use the block.
__global__ __launch_bounds__(256) void slabfill_kernel(PermuteParams p) {
    const int P = p.totals[0];
    const int lane = lane_id();
    for (int base = blockIdx.x * blockDim.x; base < P; base += gridDim.x * blockDim.x) {
        const int pr = base + threadIdx.x;
        const bool act = pr < P;
        const int e = act ? p.pair_expert[pr] : -1;
        const uint64_t m = act ? p.pair_mask[pr] : 0ull;
        uint64_t todo = ballot(act);
        while (todo) {
            const int leader = __ffsll((long long)todo) - 1;
            const int ecur = __shfl(e, leader);
            const bool mine = act && (e == ecur);
            todo &= ~ballot(mine);
            for (int c = 0; c < p.B; ++c) {
                const bool use = mine && ((m >> c) & 1ull);
                const uint64_t bits = ballot(use);
                if (!bits) continue;
                int slot = 0;
                if (lane == leader) slot = atomicAdd(&p.slab_cursor[ecur * p.B + c], __popcll(bits));
                slot = __shfl(slot, leader);
                if (use) p.slab_rows[slot + __popcll(bits & lanes_below())] = pr;
            }
        }
    }
}

}  // namespace unifmoe
