// Fused routing kernel (Sec. III-B and III-C): router logits, shared demand,
// shared block count and prototype selection, residual softmax, sort,
// cumulative-mass expert count, and the per-tile counts that the
// permutation needs.
//
// Phase 1 computes the 1 + K + B logits of each token (x W_shr, x W_1..x W_K,
// x mu_1..x mu_B) into LDS:
//   * bf16 tokens: x W_1.., x mu_1.. on the matrix cores. The fp32 router
//     and prototype weights are pre-split into three bf16 parts (hi + mid +
//     lo carries all 24 significand bits), so every bf16 x bf16 product is
//     exact and only the fp32 accumulation order differs from a sequential
//     dot product. x W_shr is an fp32 dot product on the vector units.
//   * fp32 tokens: sequential fp32 FMA dot products.
// Phase 2 decides each token with a group of 16, 32 or 64 lanes (one lane
// per expert and per block) using wave-level exchanges: a butterfly maximum
// and index-order broadcast sums for the softmax, broadcast comparisons for
// the rankings (ties toward the lower index), a lane permute for the sort
// and an in-order prefix with a ballot for the cumulative-mass count. Every
// step is the paper's order in fp32 with explicitly rounded operations.
// Per tile of 64 tokens, the rows per (expert, block) slab and the pairs per
// expert are counted in LDS and written out for the permutation.
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kRouteTok = 128;
// 4 waves: in the logits, wave w takes tokens 64 (w & 1).. and half (w >> 1)
// of the k range; then all four share each tile's decisions.
constexpr int kRouteThreads = 256;

struct RouteParams {
    int N, d, K, B, NL, NLP, lstride, key_bits;
    float tau, one_minus_2tau, t_mass, alpha_fixed;
    int max_shared, alpha_mode, mass_mode, fixed_k, select_mode;
    const void* X;
    const uint8_t* valid;
    const float* Wr;    // fp32 logits: [K+1][d]
    const float* mu;    // fp32 logits: [B][d]
    const u16* Wsplit;  // bf16 logits: [3][NLP][d], rows W_1..W_K, mu_1..mu_B, 0...
    float* alpha;
    int* nsh;
    uint64_t* mask;
    int* nres;
    int* eids;
    float* wts;
    int* bin_count;   // [kBinCopies][(K+1) << key_bits] pairs per (expert, mask key), or null
    int* tile_cnt;    // [ceil(N / kTileTok)][(K+1) B + K+1]: per tile of tokens, rows per (expert, block)
                      // slab, then pairs per expert; or null
    int* exp_total;   // [kExpCopies][K+1] pairs per expert (tile i adds into copy i % kExpCopies)
    int* pair_rank;   // [N][K+1]: slot of each pair within its bin copy
    // Copy job carried by the decisions launch (forward of bf16 layers): the
    // last cvt_blocks workgroups convert cvt_n8 16-byte chunks of bf16 at
    // cvt_src to fp16 at cvt_dst (bf16_to_f16_chunks). The decisions are
    // bound by latency and leave HBM bandwidth idle, which the copy uses.
    const u16* cvt_src;
    u16* cvt_dst;
    size_t cvt_n8;
    int cvt_blocks;
};

// bf16 -> fp16 of chunks [i0, n8) with stride `stride` (16-byte chunks of 8
// values). Each value is rounded to nearest even (exact for bf16 magnitudes
// in [2^-17, 65504]; larger ones become infinities). Four chunks per pass are
// loaded before any is converted, so each thread keeps four loads in flight.
__device__ __forceinline__ void bf16_to_f16_chunks(const u16* __restrict__ src, u16* __restrict__ dst, size_t n8,
                                                   size_t i0, size_t stride) {
    constexpr int U = 4;
    for (size_t i = i0; i < n8; i += U * stride) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (i + u * stride < n8) v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src) + i + u * stride);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (i + u * stride < n8) {
                u32x4 o;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    o[q] = pack_f16x2(__uint_as_float(v[u][q] << 16), __uint_as_float(v[u][q] & 0xffff0000u));
                reinterpret_cast<u32x4*>(dst)[i + u * stride] = o;
            }
        }
    }
}

// The copy role of a routing launch: true (after doing its share of the
// copy) for the last p.cvt_blocks workgroups of the grid.
__device__ __forceinline__ bool route_copy_role(const RouteParams& p) {
    const int first = (int)gridDim.x - p.cvt_blocks;
    if ((int)blockIdx.x < first) return false;
    bf16_to_f16_chunks(p.cvt_src, p.cvt_dst, p.cvt_n8, (size_t)(blockIdx.x - first) * blockDim.x + threadIdx.x,
                       (size_t)p.cvt_blocks * blockDim.x);
    return true;
}

// Exact three-way split of an fp32 value into bf16 parts, in workgroups
// [0, nsplit); the workgroups after them zero zwords words at zero (the
// forward's counters, in the same launch).
__global__ void split_router_kernel(const float* __restrict__ Wr, const float* __restrict__ mu,
                                    int K, int B, int d, int NLP, u16* __restrict__ out, int nsplit,
                                    uint32_t* __restrict__ zero, size_t zwords) {
    if ((int)blockIdx.x >= nsplit) {
        const size_t stride = (size_t)(gridDim.x - nsplit) * blockDim.x;
        for (size_t i = (size_t)(blockIdx.x - nsplit) * blockDim.x + threadIdx.x; i < zwords; i += stride)
            zero[i] = 0u;
        return;
    }
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int total = NLP * d;
    if (i >= total) return;
    const int j = i / d, k = i - (i / d) * d;
    float w = 0.f;
    if (j < K) w = Wr[(size_t)(j + 1) * d + k];
    else if (j < K + B) w = mu[(size_t)(j - K) * d + k];
    const u16 hi = f2bf(w);
    const float r1 = w - bf2f(hi);
    const u16 mid = f2bf(r1);
    const float r2 = r1 - bf2f(mid);
    out[i] = hi;
    out[total + i] = mid;
    out[2 * total + i] = f2bf(r2);
}

// Logits of the bf16 path. Each wave takes 64 tokens (four 16-row MFMA
// fragments), so every weight fragment it loads serves four MFMAs.
//  * The K + B expert and prototype logits run on the matrix cores in NCT
//    16-column tiles, three exact bf16 parts per weight.
//  * The shared-demand logit x W_shr is a plain fp32 dot product on the
//    vector units, in the shadow of the MFMAs: each lane sums its 8 k of
//    every k step, then the four lane groups of a row are added.
// Every operand of a k step is loaded together, D - 1 k steps ahead of its
// use, so the loads overlap each other and the MFMAs of earlier steps.
template <int NCT>
__device__ __forceinline__ void route_logits_bf16(const RouteParams& p, float* L, int tok0) {
    constexpr int RT = 4;                    // 16-row fragments per wave
    constexpr int D = (NCT <= 2) ? 3 : 2;    // register sets in the ring
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int w = wave & 1, kh = wave >> 1;  // token half, k half
    const u16* X = static_cast<const u16*>(p.X);
    f32x4 acc[RT][NCT];
    float sh[RT];
#pragma unroll
    for (int i = 0; i < RT; ++i) {
        sh[i] = 0.f;
#pragma unroll
        for (int j = 0; j < NCT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const int kof = (lane >> 4) * 8;
    const u16* xr[RT];
#pragma unroll
    for (int i = 0; i < RT; ++i) {
        // Rows past N read row N - 1; their logits are never used.
        const int r = min(tok0 + w * 64 + i * 16 + (lane & 15), p.N - 1);
        xr[i] = X + (size_t)r * p.d + kof;
    }
    const u16* wb = p.Wsplit + (size_t)(lane & 15) * p.d + kof;
    const float* wsh = p.Wr + kof;           // row 0 of the fp32 router: W_shr
    const size_t part_stride = (size_t)p.NLP * p.d, ct_stride = (size_t)16 * p.d;
    const int nks_all = p.d / 32;
    const int ks0 = kh ? nks_all / 2 : 0;
    const int nks = kh ? nks_all - nks_all / 2 : nks_all / 2;
    struct Set {
        u32x4 a[RT], b[3][NCT], s0, s1;
    };
    Set ring[D];
    auto load = [&](int ks, Set& S) {
        const int k0 = (ks0 + ks) * 32;
#pragma unroll
        for (int i = 0; i < RT; ++i) S.a[i] = ld16(xr[i] + k0);
#pragma unroll
        for (int part = 0; part < 3; ++part)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) S.b[part][ct] = ld16(wb + part * part_stride + ct * ct_stride + k0);
        S.s0 = ld16(wsh + k0);
        S.s1 = ld16(wsh + k0 + 4);
    };
    auto compute = [&](const Set& S) {
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
            for (int part = 0; part < 3; ++part) {
                const bf16x8 b = as_bf16x8(S.b[part][ct]);
#pragma unroll
                for (int i = 0; i < RT; ++i) acc[i][ct] = mfma16x16x32(as_bf16x8(S.a[i]), b, acc[i][ct]);
            }
#pragma unroll
        for (int i = 0; i < RT; ++i) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t u = S.a[i][q];
                sh[i] = fmaf(__uint_as_float(u << 16), __uint_as_float(q < 2 ? S.s0[2 * q] : S.s1[2 * q - 4]), sh[i]);
                sh[i] = fmaf(__uint_as_float(u & 0xffff0000u),
                             __uint_as_float(q < 2 ? S.s0[2 * q + 1] : S.s1[2 * q - 3]), sh[i]);
            }
        }
    };
#pragma unroll
    for (int i = 0; i < D - 1; ++i)
        if (i < nks) load(i, ring[i]);
    for (int ks = 0; ks < nks; ks += D) {
#pragma unroll
        for (int i = 0; i < D; ++i) {
            if (ks + i < nks) {
                if (ks + i + D - 1 < nks) load(ks + i + D - 1, ring[(i + D - 1) % D]);
                compute(ring[i]);
            }
        }
    }
    // Column 0: the shared-demand logit; columns 1..: the MFMA tiles. The
    // second k half is written first; the first adds it to its own sums
    // (same order for every token).
#pragma unroll
    for (int i = 0; i < RT; ++i) {
        float v = sh[i];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        sh[i] = v;
    }
    for (int half = 1; half >= 0; --half) {
        if (kh == half) {
#pragma unroll
            for (int i = 0; i < RT; ++i) {
                float* row0 = L + (size_t)(w * 64 + i * 16) * p.lstride;
                if (lane < 16) {
                    float* d0 = row0 + lane * p.lstride;
                    *d0 = half ? sh[i] : sh[i] + *d0;
                }
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        float* d = row0 + ((lane >> 4) * 4 + r) * p.lstride + 1 + ct * 16 + (lane & 15);
                        *d = half ? acc[i][ct][r] : acc[i][ct][r] + *d;
                    }
            }
        }
        __syncthreads();
    }
}

__device__ __forceinline__ void route_logits_f32(const RouteParams& p, float* L, int tok0) {
    const float* X = static_cast<const float*>(p.X);
    for (int idx = threadIdx.x; idx < kRouteTok * p.NL; idx += blockDim.x) {
        const int t = idx / p.NL, j = idx - (idx / p.NL) * p.NL, tok = tok0 + t;
        if (tok >= p.N) continue;
        const float* w = (j <= p.K) ? p.Wr + (size_t)j * p.d : p.mu + (size_t)(j - 1 - p.K) * p.d;
        const float* x = X + (size_t)tok * p.d;
        float s = 0.f;
        for (int i = 0; i < p.d; ++i) s = fmaf(x[i], w[i], s);
        L[t * p.lstride + j] = s;
    }
}

// Total-order key of a float for ranking: for non-NaN values it orders as
// the float comparison does (-0 is first mapped to +0, so the two tie), and
// a NaN gets a fixed place, so ranks computed with it always form a
// permutation, whatever the inputs hold.
__device__ __forceinline__ uint32_t rank_key(float f) {
    const uint32_t u = __float_as_uint(f + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Tokens are decided in tiles of kTileTok (one wave's ballot); the
// permutation's per-tile counts use the same tiles.
constexpr int kTileTok = 64;

// Lanes per token in the decisions: the smallest power of two >= max(K, B),
// at least 16.
__host__ __device__ __forceinline__ int decide_lanes(int K, int B) {
    const int n = K > B ? K : B;
    return n <= 16 ? 16 : (n <= 32 ? 32 : 64);
}

// Decisions of Sec. III-B and III-C for 64 / L tokens of one tile per call,
// L lanes per token (lane j of a token's group stands for expert j + 1 and
// block j), with wave-level exchanges instead of per-token loops:
//   alpha, b          every lane of the group, from the shared logit
//   I_shr             lane c ranks x mu_c against the other B priorities
//                     (broadcasts in index order, ties to the lower index)
//   softmax           group maximum (butterfly), then the sum of the
//                     exponentials in index order (broadcasts), fp32
//   q, p              lane j ranks s_j; a permute sends (s_j, j + 1) to lane
//                     rank(j), so lane r then holds p_r and q_r
//   P_r, k            lane r sums p_0..p_r in order; k is the first lane
//                     whose prefix reaches the target (ballot), else K
// All arithmetic is the paper's order in fp32 with explicitly rounded
// operations. `row` is the token's logit row in LDS (shared logit, K expert
// logits, B priorities); `t` the token's index in the tile (tokens at or past
// `ntok` are outside the layer and write nothing); `cnt` the tile's LDS
// counters (rows per (expert, block) slab, then pairs per expert), or null.
template <int L>
__device__ __forceinline__ void decide_group(const RouteParams& p, const float* row, int tok0, int t, int ntok,
                                             bool tok_valid, int* cnt) {
    static_assert(L == 16 || L == 32 || L == 64, "lane groups");
    const int K = p.K, B = p.B;
    const int lane = lane_id(), j = lane & (L - 1), gbase = lane - j;
    const int tok = tok0 + t;
    const bool in_range = t < ntok;
    const bool v = in_range && tok_valid;
    const uint64_t gmask = (L == 64) ? ~0ull : ((1ull << L) - 1ull);
    auto group_bits = [&](bool pred) { return (ballot(pred) >> gbase) & gmask; };

    // Eq. alpha (adaptive) or the fixed-alpha ablation.
    float alpha;
    if (p.alpha_mode == 0) {
        const float sig = __fdiv_rn(1.0f, __fadd_rn(1.0f, expf(-row[0])));
        alpha = __fadd_rn(p.tau, __fmul_rn(p.one_minus_2tau, sig));
    } else {
        alpha = p.alpha_fixed;
    }
    // Eq. block-count, half to even; clamp to [1, B-1] (adaptive), cap.
    // (fminf/fmaxf drop a NaN alpha, so b stays in range for any input.)
    int b = (int)rintf(fminf(fmaxf(__fmul_rn((float)B, alpha), 0.0f), (float)B));
    if (p.alpha_mode == 0) b = min(max(b, 1), B - 1);
    b = min(b, p.max_shared);

    // Eq. block-priority / shared-indices: block j is shared when fewer than
    // b priorities come before it (decreasing, ties to the lower index).
    bool shared;
    if (p.select_mode == 0) {
        const uint32_t uk = j < B ? rank_key(row[1 + K + j]) : 0u;
        int ru = 0;
#pragma unroll 16
        for (int c = 0; c < L; ++c) {
            const uint32_t o = (uint32_t)__shfl((int)uk, gbase + c);
            ru += (o > uk) || (o == uk && c < j);
        }
        shared = j < B && ru < b;
    } else {
        shared = j < b;
    }
    const uint64_t mask = group_bits(shared);

    // Eq. residual-router-score: max-subtracted softmax, index-order sum.
    const float l = j < K ? row[1 + j] : -INFINITY;
    float m = l;
#pragma unroll
    for (int o = L / 2; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    const float e = j < K ? expf(__fsub_rn(l, m)) : 0.f;
    float S = 0.f;
#pragma unroll 16
    for (int c = 0; c < L; ++c) {
        const float o = __shfl(e, gbase + c);
        if (c < K) S = __fadd_rn(S, o);
    }
    const float s = __fdiv_rn(e, S);
    // Eq. sorted-affinity: ranks by decreasing affinity, ties to the lower
    // index; padding lanes (j >= K) rank after every expert, so the ranks of
    // the group are a permutation of 0..L-1.
    const uint32_t sk = j < K ? rank_key(s) : 0u;
    int rs = 0;
#pragma unroll 16
    for (int c = 0; c < L; ++c) {
        const uint32_t o = (uint32_t)__shfl((int)sk, gbase + c);
        rs += (o > sk) || (o == sk && c < j);
    }
    const int dst = (gbase + rs) << 2;
    const float ps = __int_as_float(__builtin_amdgcn_ds_permute(dst, __float_as_int(s)));
    const int qs = __builtin_amdgcn_ds_permute(dst, j + 1);
    // Eq. beta / expert-count: the smallest prefix reaching the target.
    int k;
    if (p.mass_mode == 2) {
        k = p.fixed_k;
    } else {
        const float beta = __fsub_rn(1.0f, alpha);
        const float target = (p.mass_mode == 0) ? fminf(beta, p.t_mass) : p.t_mass;
        float P = 0.f;
#pragma unroll 16
        for (int c = 0; c < L; ++c) {
            const float o = __shfl(ps, gbase + c);
            if (c <= j && c < K) P = __fadd_rn(P, o);
        }
        const uint64_t reached = group_bits(j < K && P >= target);
        k = reached ? __builtin_ctzll(reached) + 1 : K;
    }

    if (in_range) {
        if (j == 0) {
            p.alpha[tok] = v ? alpha : 0.f;
            p.nsh[tok] = v ? b : 0;
            p.mask[tok] = v ? mask : 0ull;
            p.nres[tok] = v ? k : 0;
        }
        if (j < K) {
            p.eids[(size_t)tok * K + j] = v ? qs : -1;
            p.wts[(size_t)tok * K + j] = v ? ps : 0.f;
        }
    }
    if (p.bin_count == nullptr) return;

    // Pairs per (expert, key of the pair's block mask): one shared pair and
    // k residual pairs per valid token. The count a bin copy had before a
    // pair adds itself is the pair's slot within that copy (pair_rank), so
    // the scatter needs no atomics; slots inside a bin follow the order the
    // atomics land in, and no result depends on it (every GEMM row is
    // computed from its own pair).
    const uint64_t full = (B == 64) ? ~0ull : ((1ull << B) - 1ull);
    const int kb = p.key_bits;
    const int ks = mask_key(mask, B, kb), kr = mask_key(~mask & full, B, kb);
    const int bc = (tok / kTileTok) % kBinCopies, nbin = (K + 1) << kb;
    // Both atomics are issued before either slot is stored (one round trip).
    int* rank = p.pair_rank + (size_t)(v ? tok : 0) * (K + 1);
    int r0 = 0, r1 = 0;
    if (v && j == 0) r0 = atomicAdd(&p.bin_count[bin_counter(ks, bc, nbin)], 1);
    if (v && j < k) r1 = atomicAdd(&p.bin_count[bin_counter((qs << kb) + kr, bc, nbin)], 1);
    if (v && j == 0) rank[0] = r0;
    if (v && j < k) rank[1 + j] = r1;
    if (cnt == nullptr) return;
    // The tile's counts: pairs per expert, and rows per slab (the shared
    // expert on I_shr, each selected residual expert on I_res). Lane c adds
    // block c's rows.
    int* ecnt = cnt + (K + 1) * B;
    if (v && j == 0) atomicAdd(&ecnt[0], 1);
    if (v && j < k) atomicAdd(&ecnt[qs], 1);
    if (v && j < B && shared) atomicAdd(&cnt[j], 1);
    int kmax = v ? k : 0;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) kmax = max(kmax, __shfl_xor(kmax, o));
    for (int i = 0; i < kmax; ++i) {
        const int ei = __shfl(qs, gbase + i);
        if (v && i < k && j < B && !shared) atomicAdd(&cnt[ei * B + j], 1);
    }
}

// Every token of a tile of kTileTok tokens whose logit rows are at `rows`
// (stride lstride): the waves [w0, w0 + nw) of the workgroup share the
// tile's tokens, 64 / L per pass.
template <int L>
__device__ __forceinline__ void decide_tile(const RouteParams& p, const float* rows, const int* vflags, int tok0,
                                            int ntok, int wave, int w0, int nw, int* cnt) {
    constexpr int TPP = 64 / L;   // tokens per wave pass
    const int g = lane_id() / L;
    for (int t0 = (wave - w0) * TPP; t0 < kTileTok; t0 += nw * TPP) {
        const int t = t0 + g;
        decide_group<L>(p, rows + (size_t)(t < ntok ? t : 0) * p.lstride, tok0, t, ntok, vflags[t] != 0, cnt);
    }
}

// The valid flags of a tile's tokens into LDS (1 for every token without a
// mask; tokens past the layer read 0): the decisions then read them without
// a global load in each pass. Called by every thread; a barrier follows.
__device__ __forceinline__ void stage_valid(const RouteParams& p, int tok0, int* vflags) {
    for (int t = threadIdx.x; t < kTileTok; t += blockDim.x) {
        const int tok = tok0 + t;
        vflags[t] = (tok < p.N) ? (p.valid == nullptr ? 1 : (int)p.valid[tok]) : 0;
    }
}

// The workgroup's tile counters (ncnt words per tile, in LDS) out to memory
// once its tiles are decided: tile i of the workgroup is layer tile
// tile0 + i * stride. Called by every thread after a barrier.
__device__ __forceinline__ void flush_counts(const RouteParams& p, const int* cnt, int ntiles, int ncnt, int tile0,
                                             int stride) {
    const int nslab = (p.K + 1) * p.B;
    for (int x = threadIdx.x; x < ncnt; x += blockDim.x)
        for (int i = 0; i < ntiles; ++i) {
            const int tile = tile0 + i * stride, c = cnt[i * ncnt + x];
            p.tile_cnt[(size_t)tile * ncnt + x] = c;
            // Pairs per expert also into the totals (few atomics, spread).
            if (x >= nslab && c) atomicAdd(&p.exp_total[(tile % kExpCopies) * (p.K + 1) + x - nslab], c);
        }
}

// The decisions of one tile with the lane count of the layer (see
// decide_lanes).
__device__ __forceinline__ void decide_tile_any(const RouteParams& p, const float* rows, const int* vflags, int tok0,
                                                int ntok, int wave, int w0, int nw, int* cnt) {
    switch (decide_lanes(p.K, p.B)) {
        case 16: decide_tile<16>(p, rows, vflags, tok0, ntok, wave, w0, nw, cnt); break;
        case 32: decide_tile<32>(p, rows, vflags, tok0, ntok, wave, w0, nw, cnt); break;
        default: decide_tile<64>(p, rows, vflags, tok0, ntok, wave, w0, nw, cnt); break;
    }
}

// NCT: 16-column logit tiles of the bf16 path (1 + K + B <= 16 NCT); 0 for
// fp32 tokens. One workgroup of 4 waves per kRouteTok tokens (two tiles):
// the logits of all of them, then the two tiles' decisions, all 4 waves on
// each tile. The last p.cvt_blocks workgroups do the launch's copy job.
template <int NCT>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(RouteParams p) {
    constexpr int NT = kRouteTok / kTileTok;
    if (route_copy_role(p)) return;
    extern __shared__ float lds_route[];
    float* L = lds_route;
    const int ncnt = (p.K + 1) * p.B + p.K + 1;
    int* cnt = reinterpret_cast<int*>(L + kRouteTok * p.lstride);   // [NT][ncnt]
    int* vflags = cnt + NT * ncnt;                                   // [NT][kTileTok]
    const int tok0 = blockIdx.x * kRouteTok;
    const bool counting = p.tile_cnt != nullptr;
    if (counting)
        for (int i = threadIdx.x; i < NT * ncnt; i += blockDim.x) cnt[i] = 0;
    for (int h = 0; h < NT; ++h) stage_valid(p, tok0 + h * kTileTok, vflags + h * kTileTok);
    if constexpr (NCT > 0) route_logits_bf16<NCT>(p, L, tok0);
    else route_logits_f32(p, L, tok0);
    __syncthreads();
    const int wave = threadIdx.x >> 6;
    int nt = 0;
    for (int h = 0; h < NT; ++h) {
        const int t0 = tok0 + h * kTileTok;
        if (t0 >= p.N) break;
        decide_tile_any(p, L + (size_t)h * kTileTok * p.lstride, vflags + h * kTileTok, t0, min(kTileTok, p.N - t0),
                        wave, 0, kRouteThreads / 64, counting ? cnt + h * ncnt : nullptr);
        ++nt;
    }
    if (counting) {
        __syncthreads();
        flush_counts(p, cnt, nt, ncnt, tok0 / kTileTok, 1);
    }
}

// Logits of bf16 tokens when the router fits in registers (1 + K + B <= 32
// columns, d <= 1024), persistent: one workgroup of 8 waves takes the 64-token
// tiles blockIdx.x, blockIdx.x + gridDim.x, ... Wave w owns k steps
// [w nks / 8, (w + 1) nks / 8) and keeps the router's three bf16 parts and
// W_shr for them in registers for all its tiles, so only token rows stream
// from memory (the next tile's rows load while this tile's partial logits
// are reduced); the 8 partial sets are summed in a fixed order and each
// token's 1 + 16 NCT logits written to logits[N][1 + 16 NCT]. The decisions
// run in route_decide_kernel.
constexpr int kRpTok = kTileTok;
constexpr int kRpWaves = 8;
constexpr int kRpThreads = kRpWaves * 64;

template <int NCT, int KPW>
__global__ __launch_bounds__(kRpThreads) void route_logits_kernel(RouteParams p, float* __restrict__ logits) {
    constexpr int RT = kRpTok / 16;          // 16-row fragments per tile
    constexpr int ncols = 1 + 16 * NCT;
    extern __shared__ float lds_route[];
    const int ls = p.lstride;
    float* Pbuf = lds_route;                                     // [8][64][ls] partial logits
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ntile_all = (p.N + kRpTok - 1) / kRpTok;
    const int nt = (ntile_all - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;

    // This wave's k steps (32 deep) and the router parts for them.
    const int nks = p.d / 32;
    const int kb = wave * nks / kRpWaves, kn = (wave + 1) * nks / kRpWaves - kb;   // kn <= KPW
    const int kof = (lane >> 4) * 8;
    const u16* wb = p.Wsplit + (size_t)(lane & 15) * p.d + kof;
    const size_t part_stride = (size_t)p.NLP * p.d, ct_stride = (size_t)16 * p.d;
    u32x4 W[KPW][3][NCT], S0[KPW], S1[KPW];
#pragma unroll
    for (int j = 0; j < KPW; ++j) {
        const int k0 = (kb + (j < kn ? j : 0)) * 32;
#pragma unroll
        for (int part = 0; part < 3; ++part)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) W[j][part][ct] = ld16(wb + part * part_stride + ct * ct_stride + k0);
        S0[j] = ld16(p.Wr + kof + k0);
        S1[j] = ld16(p.Wr + kof + k0 + 4);
    }
    const u16* X = static_cast<const u16*>(p.X);
    u32x4 xa[KPW][RT];
    auto load_x = [&](int i) {
        const int tok0 = ((int)blockIdx.x + i * (int)gridDim.x) * kRpTok;
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            // Rows past N read row N - 1; their logits are never written.
            const u16* xr = X + (size_t)min(tok0 + r * 16 + (lane & 15), p.N - 1) * p.d + kof;
#pragma unroll
            for (int j = 0; j < KPW; ++j) xa[j][r] = ld16(xr + (kb + (j < kn ? j : 0)) * 32);
        }
    };
    if (nt > 0) load_x(0);
    for (int i = 0; i < nt; ++i) {
        const int tok0 = ((int)blockIdx.x + i * (int)gridDim.x) * kRpTok;
        f32x4 acc[RT][NCT];
        float sh[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            sh[r] = 0.f;
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) acc[r][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int j = 0; j < KPW; ++j) {
            if (j < kn) {
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int part = 0; part < 3; ++part)
#pragma unroll
                        for (int r = 0; r < RT; ++r)
                            acc[r][ct] = mfma16x16x32(as_bf16x8(xa[j][r]), as_bf16x8(W[j][part][ct]), acc[r][ct]);
#pragma unroll
                for (int r = 0; r < RT; ++r)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint32_t u = xa[j][r][q];
                        sh[r] = fmaf(__uint_as_float(u << 16), __uint_as_float(q < 2 ? S0[j][2 * q] : S1[j][2 * q - 4]), sh[r]);
                        sh[r] = fmaf(__uint_as_float(u & 0xffff0000u),
                                     __uint_as_float(q < 2 ? S0[j][2 * q + 1] : S1[j][2 * q - 3]), sh[r]);
                    }
            }
        }
        // The next tile's rows are in flight during the reduction.
        if (i + 1 < nt) load_x(i + 1);
        // This wave's partial logits: column 0 the shared demand, columns
        // 1.. the MFMA tiles. (The barrier after the previous tile's sum
        // orders its reads of Pbuf before these writes.)
        float* P = Pbuf + wave * kRpTok * ls;
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            float v = sh[r];
            v += __shfl_xor(v, 16);
            v += __shfl_xor(v, 32);
            if (lane < 16) P[(r * 16 + lane) * ls] = v;
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    P[(r * 16 + (lane >> 4) * 4 + e) * ls + 1 + ct * 16 + (lane & 15)] = acc[r][ct][e];
        }
        lds_barrier();
        // Sum of the 8 k slices, in wave order, straight to memory.
        const int ntok = min(kRpTok, p.N - tok0);
        for (int e = tid; e < ntok * ncols; e += blockDim.x) {
            const int t = e / ncols, c = e - t * ncols;
            float v = 0.f;
#pragma unroll
            for (int w = 0; w < kRpWaves; ++w) v += Pbuf[(w * kRpTok + t) * ls + c];
            logits[(size_t)tok0 * ncols + e] = v;
        }
        lds_barrier();
    }
}

// Decisions of one 64-token tile per workgroup of NW waves (L lanes per
// token, see decide_lanes), from the logits route_logits_kernel wrote (ncols
// per token), staged in LDS rows; then the tile's counters out to memory.
// The last p.cvt_blocks workgroups do the launch's copy job instead. With
// few tiles (up to two per compute unit) 8 waves share a tile, so each wave
// runs half the passes of dependent lane exchanges; with more tiles 4 do,
// which leaves room on each compute unit for more tiles and the copy.
template <int L, int NW>
__global__ __launch_bounds__(NW * 64) void route_decide_kernel(RouteParams p, const float* __restrict__ logits,
                                                               int ncols) {
    if (route_copy_role(p)) return;
    extern __shared__ float lds_dec[];
    const int ls = p.lstride;
    float* rows = lds_dec;                                       // [64][ls]
    const int ncnt = (p.K + 1) * p.B + p.K + 1;
    int* cnt = reinterpret_cast<int*>(rows + kTileTok * ls);     // the tile's counters
    int* vflags = cnt + ncnt;                                    // [kTileTok] valid flags
    const bool counting = p.tile_cnt != nullptr;
    const int tile = blockIdx.x, tok0 = tile * kTileTok, ntok = min(kTileTok, p.N - tok0);
    // The tokens' valid flags are loaded first and stored after the logit
    // rows' batch, so their latencies overlap.
    const int tv = (int)threadIdx.x;
    uint32_t vb = 1u;
    if (tv < ntok && p.valid != nullptr) vb = p.valid[tok0 + tv];
    batched_copy(
        ntok * ncols, [&](int e) { return logits[(size_t)tok0 * ncols + e]; },
        [&](int e, float v) {
            const int t = e / ncols;
            rows[t * ls + e - t * ncols] = v;
        });
    asm volatile("" : "+v"(vb));   // the byte is first used here, after the rows' batch
    if (tv < kTileTok) vflags[tv] = (tv < ntok && vb != 0u) ? 1 : 0;
    if (counting)
        for (int i = threadIdx.x; i < ncnt; i += blockDim.x) cnt[i] = 0;
    __syncthreads();
    decide_tile<L>(p, rows, vflags, tok0, ntok, (int)threadIdx.x >> 6, 0, NW, counting ? cnt : nullptr);
    if (counting) {
        __syncthreads();
        flush_counts(p, cnt, 1, ncnt, tile, 1);
    }
}

}  // namespace unifmoe
