// Fused routing kernel (Sec. III-B and III-C): router logits, shared demand,
// shared block count and prototype selection, residual softmax, sort,
// cumulative-mass expert count, and the per-(expert, block) counts that the
// permutation needs.
//
// One workgroup of two waves routes 128 tokens. Phase 1 computes the
// 1 + K + B logits of each token (x W_shr, x W_1..x W_K, x mu_1..x mu_B)
// into LDS:
//   * bf16 tokens: x W_1.., x mu_1.. on the matrix cores. The fp32 router
//     and prototype weights are pre-split into three bf16 parts (hi + mid +
//     lo carries all 24 significand bits), so every bf16 x bf16 product is
//     exact and only the fp32 accumulation order differs from a sequential
//     dot product. x W_shr is an fp32 dot product on the vector units.
//   * fp32 tokens: sequential fp32 FMA dot products.
// Phase 2 takes one token per lane and runs the decisions in the paper's
// order in fp32 with explicitly rounded operations; ties break toward the
// lower index. The per-(expert, block) row counts are gathered with wave
// ballots into LDS, then added to global memory once per workgroup.
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kRouteTok = 128;
// 4 waves: in the logits, wave w takes tokens 64 (w & 1).. and half (w >> 1)
// of the k range; then waves 0 and 1 take one token per thread.
constexpr int kRouteThreads = 256;

struct RouteParams {
    int N, d, K, B, NL, NLP, lstride, key_bits;
    int key_stride;     // words per token of the LDS ranking keys, 0 if none
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
    int* bin_count;   // [(K+1) << key_bits] pairs per (expert, mask key), or null
    int* slab_count;  // [kSlabCopies][(K+1) B + K+1]: rows per (expert, block), then pairs per expert; or null
    int* pair_rank;   // [N][K+1]: slot of each pair within its (expert, key) bin (with bin_count)
};

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

// Words per token of the ranking keys: max(K, B) rounded up to 4.
__host__ __device__ __forceinline__ int key_row(int K, int B) { return ((K > B ? K : B) + 3) & ~3; }

// Total-order key of a float for ranking: for non-NaN values it orders as
// the float comparison does (-0 is first mapped to +0, so the two tie), and
// a NaN gets a fixed place, so ranks computed with it always form a
// permutation, whatever the inputs hold.
__device__ __forceinline__ uint32_t rank_key(float f) {
    const uint32_t u = __float_as_uint(f + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Rank of entry j among the n keys of a row (16-byte aligned, zero-padded to
// a multiple of 4): the number of entries that come before it in decreasing
// key order, ties to the lower index. Padding keys are 0 and sit at indices
// >= n, so they never come first.
__device__ __forceinline__ int rank_in_row(const uint32_t* keys, int n, int j) {
    const uint32_t kj = keys[j];
    int rank = 0;
    for (int c = 0; c < n; c += 4) {
        const u32x4 k4 = *reinterpret_cast<const u32x4*>(keys + c);
#pragma unroll
        for (int q = 0; q < 4; ++q) rank += (k4[q] > kj) || (k4[q] == kj && c + q < j);
    }
    return rank;
}

// The same from the float values (no key row).
__device__ __forceinline__ int rank_in_values(const float* v, int n, int j) {
    const uint32_t kj = rank_key(v[j]);
    int rank = 0;
    for (int c = 0; c < n; ++c) {
        const uint32_t kc = rank_key(v[c]);
        rank += (kc > kj) || (kc == kj && c < j);
    }
    return rank;
}

constexpr int kRankBatch = 8;   // residual-pair atomics in flight per token

// Rankings of at most this many entries run on registers.
constexpr int kSmallRank = 16;

// Decisions for token tok0 + tid, one token per lane of whole waves (the
// counting below merges the lanes of a wave).
__device__ __forceinline__ void route_decide(const RouteParams& p, float* L, float* PS, int* QS, uint32_t* KEYS,
                                             int* slab_lds, int tok0, int tid) {
    const int K = p.K, B = p.B, tok = tok0 + tid;
    const bool in_range = tok < p.N;
    const bool v = in_range && (p.valid == nullptr || p.valid[tok] != 0);
    float* row = L + tid * p.lstride;
    float* ps = PS + tid * (K + 1);
    int* qs = QS + tid * (K + 1);
    // Ranking keys: a 16-byte-aligned row per token when the workgroup's
    // LDS has room for them (kp > 0), else ranked straight from the values.
    const int kp = p.key_stride;
    uint32_t* keys = KEYS + tid * kp;
    uint64_t mask = 0, sel = 0;
    int k = 0;
    if (v) {
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
        // Eq. block-priority / shared-indices: the b largest x mu_c.
        if (p.select_mode == 0) {
            const float* u = row + 1 + K;
            if (B <= kSmallRank) {
                // All keys in registers; padding keys 0 never come first.
                uint32_t uk[kSmallRank];
#pragma unroll
                for (int c = 0; c < kSmallRank; ++c) uk[c] = c < B ? rank_key(u[c]) : 0u;
#pragma unroll
                for (int c = 0; c < kSmallRank; ++c) {
                    int rank = 0;
#pragma unroll
                    for (int c2 = 0; c2 < kSmallRank; ++c2) rank += (uk[c2] > uk[c]) || (uk[c2] == uk[c] && c2 < c);
                    if (c < B && rank < b) mask |= 1ull << c;
                }
            } else if (kp > 0) {
                for (int c = 0; c < kp; ++c) keys[c] = c < B ? rank_key(u[c]) : 0u;
                for (int c = 0; c < B; ++c)
                    if (rank_in_row(keys, B, c) < b) mask |= 1ull << c;
            } else {
                for (int c = 0; c < B; ++c)
                    if (rank_in_values(u, B, c) < b) mask |= 1ull << c;
            }
        } else {
            mask = (b >= 64) ? ~0ull : ((1ull << b) - 1ull);
        }
        // Eq. residual-router-score: max-subtracted softmax, index-order sum.
        float* l = row + 1;
        if (K <= kSmallRank) {
            // The same steps on registers: softmax, ranks, then the sorted
            // weights back from LDS for the prefix of Eq. expert-count.
            float lv[kSmallRank];
#pragma unroll
            for (int j = 0; j < kSmallRank; ++j) lv[j] = j < K ? l[j] : 0.f;
            float m = lv[0];
#pragma unroll
            for (int j = 1; j < kSmallRank; ++j) m = j < K ? fmaxf(m, lv[j]) : m;
            float S = 0.f;
#pragma unroll
            for (int j = 0; j < kSmallRank; ++j) {
                lv[j] = j < K ? expf(__fsub_rn(lv[j], m)) : 0.f;
                S = j < K ? __fadd_rn(S, lv[j]) : S;
            }
            uint32_t ek[kSmallRank];
#pragma unroll
            for (int j = 0; j < kSmallRank; ++j) {
                lv[j] = __fdiv_rn(lv[j], S);
                ek[j] = j < K ? rank_key(lv[j]) : 0u;
            }
            int rk[kSmallRank];
#pragma unroll
            for (int j = 0; j < kSmallRank; ++j) {
                int rank = 0;
#pragma unroll
                for (int j2 = 0; j2 < kSmallRank; ++j2) rank += (ek[j2] > ek[j]) || (ek[j2] == ek[j] && j2 < j);
                rk[j] = rank;
                if (j < K) {
                    ps[rank] = lv[j];
                    qs[rank] = j + 1;
                }
            }
            if (p.mass_mode == 2) {
                k = p.fixed_k;
            } else {
                const float beta = __fsub_rn(1.0f, alpha);
                const float target = (p.mass_mode == 0) ? fminf(beta, p.t_mass) : p.t_mass;
                float sv[kSmallRank];
#pragma unroll
                for (int n = 0; n < kSmallRank; ++n) sv[n] = n < K ? ps[n] : 0.f;
                float P = 0.f;
                k = K;
                bool found = false;
#pragma unroll
                for (int n = 0; n < kSmallRank; ++n) {
                    if (n < K && !found) {
                        P = __fadd_rn(P, sv[n]);
                        if (P >= target) {
                            k = n + 1;
                            found = true;
                        }
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < kSmallRank; ++j)
                if (j < K && rk[j] < k) sel |= 1ull << j;
        } else {
        float m = l[0];
        for (int j = 1; j < K; ++j) m = fmaxf(m, l[j]);
        float S = 0.f;
        for (int j = 0; j < K; ++j) {
            const float e = expf(__fsub_rn(l[j], m));
            l[j] = e;
            S = __fadd_rn(S, e);
        }
        for (int j = 0; j < K; ++j) l[j] = __fdiv_rn(l[j], S);
        // Eq. sorted-affinity: rank by decreasing affinity, ties to lower index.
        for (int j = 0; j < kp; ++j) keys[j] = j < K ? rank_key(l[j]) : 0u;
        for (int j = 0; j < K; ++j) {
            const int rank = kp > 0 ? rank_in_row(keys, K, j) : rank_in_values(l, K, j);
            ps[rank] = l[j];
            qs[rank] = j + 1;
        }
        // Eq. beta / expert-count: smallest prefix reaching the target.
        if (p.mass_mode == 2) {
            k = p.fixed_k;
        } else {
            const float beta = __fsub_rn(1.0f, alpha);
            const float target = (p.mass_mode == 0) ? fminf(beta, p.t_mass) : p.t_mass;
            float P = 0.f;
            k = K;
            for (int n = 0; n < K; ++n) {
                P = __fadd_rn(P, ps[n]);
                if (P >= target) {
                    k = n + 1;
                    break;
                }
            }
        }
        for (int i = 0; i < k; ++i) sel |= 1ull << (qs[i] - 1);
        }
        p.alpha[tok] = alpha;
        p.nsh[tok] = b;
        p.mask[tok] = mask;
        p.nres[tok] = k;
    } else if (in_range) {
        p.alpha[tok] = 0.f;
        p.nsh[tok] = 0;
        p.mask[tok] = 0;
        p.nres[tok] = 0;
        for (int j = 0; j < K; ++j) {
            ps[j] = 0.f;
            qs[j] = -1;
        }
    }
    if (p.bin_count == nullptr) return;

    // Pairs per (expert, key of the pair's block mask): one shared pair and
    // k residual pairs per valid token.
    const uint64_t full = (B == 64) ? ~0ull : ((1ull << B) - 1ull);
    const int kb = p.key_bits;
    const int lane = lane_id();
    const uint64_t rmask = ~mask & full;
    const int ks = mask_key(mask, B, kb);
    const int kr = mask_key(rmask, B, kb);
    // The count of a bin taken before a pair adds itself is the pair's slot
    // within the bin (pair_rank), so the scatter needs no atomics. The order
    // of the slots inside a bin is whatever order the atomics land in; no
    // result depends on it (every GEMM row is computed from its own pair).
    // The shared pair's atomic and those of the first kRankBatch residual
    // pairs are issued before any result is used, so their latencies overlap.
    int* rank = p.pair_rank + (size_t)(v ? tok : 0) * (K + 1);
    const int r0 = v ? atomicAdd(&p.bin_count[ks], 1) : 0;
    for (int i0 = 0; i0 < K; i0 += kRankBatch) {
        if (!ballot(v && i0 < k)) break;
        int r[kRankBatch];
#pragma unroll
        for (int u = 0; u < kRankBatch; ++u)
            r[u] = (v && i0 + u < k) ? atomicAdd(&p.bin_count[(qs[i0 + u] << kb) + kr], 1) : 0;
#pragma unroll
        for (int u = 0; u < kRankBatch; ++u)
            if (v && i0 + u < k) rank[1 + i0 + u] = r[u];
    }
    if (v) rank[0] = r0;
    // Pairs per expert and rows per (expert, block), after the row counts in
    // slab_lds: lane c (< B) holds the ballot of the tokens whose shared
    // blocks include c, so expert e's rows on block c (the shared expert on
    // I_shr, a residual expert on I_res) are one popcount, and each expert
    // needs one LDS add per block lane.
    int* ecnt = slab_lds + (K + 1) * B;
    uint64_t mb = 0;
    for (int c = 0; c < B; ++c) {
        const uint64_t bits = ballot(v && ((mask >> c) & 1ull));
        if (lane == c) mb = bits;
    }
    const uint64_t vb = ballot(v);
    if (!vb) return;
    if (lane == 0) atomicAdd(&ecnt[0], __popcll(vb));
    if (lane < B) {
        const int n = __popcll(mb);
        if (n) atomicAdd(&slab_lds[lane], n);
    }
    for (int e = 1; e <= K; ++e) {
        const uint64_t hb = ballot(v && ((sel >> (e - 1)) & 1ull));
        if (!hb) continue;
        if (lane == 0) atomicAdd(&ecnt[e], __popcll(hb));
        if (lane < B) {
            const int n = __popcll(hb & ~mb);
            if (n) atomicAdd(&slab_lds[e * B + lane], n);
        }
    }
}

// NCT: 16-column logit tiles of the bf16 path (1 + K + B <= 16 NCT); 0 for
// fp32 tokens.
template <int NCT>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(RouteParams p) {
    extern __shared__ float lds_route[];
    float* L = lds_route;
    float* PS = L + kRouteTok * p.lstride;
    int* QS = reinterpret_cast<int*>(PS + kRouteTok * (p.K + 1));
    uint32_t* KEYS = reinterpret_cast<uint32_t*>(QS + kRouteTok * (p.K + 1));   // 16-byte aligned
    int* slab_lds = reinterpret_cast<int*>(KEYS + kRouteTok * p.key_stride);
    const int tok0 = blockIdx.x * kRouteTok;
    const int nslab = (p.K + 1) * p.B;
    // slab_lds: rows per slab, then pairs per expert.
    const int ncnt = nslab + p.K + 1;
    if (p.slab_count)
        for (int i = threadIdx.x; i < ncnt; i += blockDim.x) slab_lds[i] = 0;
    if constexpr (NCT > 0) route_logits_bf16<NCT>(p, L, tok0);
    else route_logits_f32(p, L, tok0);
    __syncthreads();
    if (threadIdx.x < kRouteTok) route_decide(p, L, PS, QS, KEYS, slab_lds, tok0, threadIdx.x);
    __syncthreads();
    // Sorted expert ids and weights of the workgroup's tokens: one contiguous
    // range of each output, written from LDS with consecutive addresses.
    {
        const int K = p.K, ntok = min(kRouteTok, p.N - tok0);
        const size_t base = (size_t)tok0 * K;
        for (int i = threadIdx.x; i < ntok * K; i += blockDim.x) {
            const int t = i / K, r = i - t * K;
            p.eids[base + i] = QS[t * (K + 1) + r];
            p.wts[base + i] = PS[t * (K + 1) + r];
        }
    }
    // Workgroup totals go to one of kSlabCopies copies of the counts, which
    // spreads the same-address atomics; the permutation sums the copies.
    if (p.slab_count) {
        int* dst = p.slab_count + (size_t)(blockIdx.x % kSlabCopies) * ncnt;
        for (int i = threadIdx.x; i < ncnt; i += blockDim.x)
            if (slab_lds[i]) atomicAdd(&dst[i], slab_lds[i]);
    }
}

// Persistent routing for bf16 tokens when the router fits in registers
// (1 + K + B <= 32 columns, d <= 768, K, B <= 16). One workgroup of 8 waves
// takes the 64-token tiles blockIdx.x, blockIdx.x + gridDim.x, ... (at most
// kRpMaxTiles). Wave w owns k steps [w nks / 8, (w + 1) nks / 8) of the
// logits and keeps the router's three bf16 parts and W_shr for them in
// registers for all its tiles, so only token rows stream from memory; each
// tile's partial logits go to LDS and are summed over the 8 k slices in a
// fixed order. Then wave i takes the decisions of tile i (one token per lane),
// the tiles' decisions running side by side.
constexpr int kRpTok = 64;
constexpr int kRpWaves = 8;
constexpr int kRpThreads = kRpWaves * 64;
constexpr int kRpMaxTiles = 4;

template <int NCT, int KPW>
__global__ __launch_bounds__(kRpThreads) void route_persist_kernel(RouteParams p) {
    constexpr int RT = kRpTok / 16;          // 16-row fragments per tile
    extern __shared__ float lds_route[];
    const int K = p.K, ls = p.lstride;
    const int ncols = 1 + 16 * NCT;
    float* Lb = lds_route;                                       // [kRpMaxTiles][64][ls]
    float* U = Lb + kRpMaxTiles * kRpTok * ls;                   // union: partials, then PS/QS
    float* Pbuf = U;                                             // [8][64][ls]
    float* PS = U;                                               // [kRpMaxTiles][64][K+1]
    int* QS = reinterpret_cast<int*>(PS + kRpMaxTiles * kRpTok * (K + 1));
    const int ufloats = max(kRpWaves * kRpTok * ls, 2 * kRpMaxTiles * kRpTok * (K + 1));
    int* slab_lds = reinterpret_cast<int*>(U + ufloats);
    const int nslab = (K + 1) * p.B, ncnt = nslab + K + 1;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ntile_all = (p.N + kRpTok - 1) / kRpTok;
    const int nt = min(kRpMaxTiles, (ntile_all - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x);
    if (p.slab_count)
        for (int i = tid; i < ncnt; i += blockDim.x) slab_lds[i] = 0;

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
            // Rows past N read row N - 1; their logits are never used.
            const u16* xr = X + (size_t)min(tok0 + r * 16 + (lane & 15), p.N - 1) * p.d + kof;
#pragma unroll
            for (int j = 0; j < KPW; ++j) xa[j][r] = ld16(xr + (kb + (j < kn ? j : 0)) * 32);
        }
    };
    if (nt > 0) load_x(0);
    for (int i = 0; i < nt; ++i) {
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
        // 1.. the MFMA tiles.
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
        // Sum of the 8 k slices, in wave order.
        float* L = Lb + i * kRpTok * ls;
        for (int e = tid; e < kRpTok * ncols; e += blockDim.x) {
            const int t = e / ncols, c = e - t * ncols;
            float v = 0.f;
#pragma unroll
            for (int w = 0; w < kRpWaves; ++w) v += Pbuf[(w * kRpTok + t) * ls + c];
            L[t * ls + c] = v;
        }
        lds_barrier();
    }
    // Decisions: wave i takes tile i (the partial buffer is reused as PS/QS).
    if (wave < nt) {
        const int tok0 = ((int)blockIdx.x + wave * (int)gridDim.x) * kRpTok;
        route_decide(p, Lb + wave * kRpTok * ls, PS + wave * kRpTok * (K + 1), QS + wave * kRpTok * (K + 1),
                     nullptr, slab_lds, tok0, lane);
    }
    __syncthreads();
    for (int i = 0; i < nt; ++i) {
        const int tok0 = ((int)blockIdx.x + i * (int)gridDim.x) * kRpTok;
        const int ntok = min(kRpTok, p.N - tok0);
        const size_t base = (size_t)tok0 * K;
        const float* ps = PS + i * kRpTok * (K + 1);
        const int* qs = QS + i * kRpTok * (K + 1);
        for (int e = tid; e < ntok * K; e += blockDim.x) {
            const int t = e / K, r = e - t * K;
            p.eids[base + e] = qs[t * (K + 1) + r];
            p.wts[base + e] = ps[t * (K + 1) + r];
        }
    }
    if (p.slab_count) {
        int* dst = p.slab_count + (size_t)(blockIdx.x % kSlabCopies) * ncnt;
        for (int i = tid; i < ncnt; i += blockDim.x)
            if (slab_lds[i]) atomicAdd(&dst[i], slab_lds[i]);
    }
}

}  // namespace unifmoe
