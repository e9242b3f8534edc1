// Fused routing kernel (Sec. III-B and III-C): router logits, shared demand,
// shared block count and prototype selection, residual softmax, sort,
// cumulative-mass expert count, and the per-(expert, block) counts that the
// permutation needs.
//
// One workgroup routes 128 tokens. Phase 1 computes the 1 + K + B logits of
// each token (x W_shr, x W_1..x W_K, x mu_1..x mu_B) into LDS:
//   * bf16 tokens: on the matrix cores. The fp32 router and prototype
//     weights are pre-split into three bf16 parts (hi + mid + lo carries all
//     24 significand bits), so every bf16 x bf16 product is exact and only
//     the fp32 accumulation order differs from a sequential dot product.
//   * fp32 tokens: sequential fp32 FMA dot products.
// Phase 2 takes one token per lane (waves 0 and 1) and runs the decisions in
// the paper's order in fp32 with explicitly rounded operations; ties break
// toward the lower index. The per-(expert, block) row counts are gathered
// with wave ballots into LDS, then added to global memory once per group.
#pragma once
#include "common.hpp"

namespace unifmoe {

constexpr int kRouteTok = 128;
constexpr int kRouteThreads = 256;
constexpr int kRouteMaxColTiles = 9;  // 1 + K + B <= 144 logits

struct RouteParams {
    int N, d, K, B, NL, NLP, lstride, key_bits;
    float tau, one_minus_2tau, t_mass, alpha_fixed;
    int max_shared, alpha_mode, mass_mode, fixed_k, select_mode;
    const void* X;
    const uint8_t* valid;
    const float* Wr;    // fp32 logits: [K+1][d]
    const float* mu;    // fp32 logits: [B][d]
    const u16* Wsplit;  // bf16 logits: [3][NLP][d], rows W_shr, W_1..W_K, mu_1..mu_B, 0...
    float* alpha;
    int* nsh;
    uint64_t* mask;
    int* nres;
    int* eids;
    float* wts;
    int* bin_count;   // [(K+1) << key_bits] pairs per (expert, mask key), or null
    int* slab_count;  // [(K+1) * B] rows per (expert, block), or null
};

// Exact three-way split of an fp32 value into bf16 parts.
__global__ void split_router_kernel(const float* __restrict__ Wr, const float* __restrict__ mu,
                                    int K, int B, int d, int NLP, u16* __restrict__ out) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int total = NLP * d;
    if (i >= total) return;
    const int j = i / d, k = i - (i / d) * d;
    float w = 0.f;
    if (j <= K) w = Wr[(size_t)j * d + k];
    else if (j <= K + B) w = mu[(size_t)(j - 1 - K) * d + k];
    const u16 hi = f2bf(w);
    const float r1 = w - bf2f(hi);
    const u16 mid = f2bf(r1);
    const float r2 = r1 - bf2f(mid);
    out[i] = hi;
    out[total + i] = mid;
    out[2 * total + i] = f2bf(r2);
}

__device__ __forceinline__ void route_logits_bf16(const RouteParams& p, float* L, int tok0) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int nct = p.NLP / 16;
    const u16* X = static_cast<const u16*>(p.X);
    f32x4 acc[2][kRouteMaxColTiles];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < kRouteMaxColTiles; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int r0 = tok0 + w * 32 + (lane & 15);
    const int r1 = r0 + 16;
    const int kof = (lane >> 4) * 8;
    for (int k0 = 0; k0 < p.d; k0 += 32) {
        u32x4 va = {0u, 0u, 0u, 0u}, vb = {0u, 0u, 0u, 0u};
        if (r0 < p.N) va = ld16(X + (size_t)r0 * p.d + k0 + kof);
        if (r1 < p.N) vb = ld16(X + (size_t)r1 * p.d + k0 + kof);
        const bf16x8 a0 = as_bf16x8(va), a1 = as_bf16x8(vb);
#pragma unroll
        for (int ct = 0; ct < kRouteMaxColTiles; ++ct) {
            if (ct < nct) {
#pragma unroll
                for (int part = 0; part < 3; ++part) {
                    const bf16x8 b = as_bf16x8(ld16(
                        p.Wsplit + (size_t)(part * p.NLP + ct * 16 + (lane & 15)) * p.d + k0 + kof));
                    acc[0][ct] = mfma16x16x32(a0, b, acc[0][ct]);
                    acc[1][ct] = mfma16x16x32(a1, b, acc[1][ct]);
                }
            }
        }
    }
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int ct = 0; ct < kRouteMaxColTiles; ++ct)
            if (ct < nct)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    L[(w * 32 + rt * 16 + (lane >> 4) * 4 + r) * p.lstride + ct * 16 + (lane & 15)] =
                        acc[rt][ct][r];
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

// Decisions for token tok0 + threadIdx.x (threads 0..127, i.e. waves 0, 1).
__device__ __forceinline__ void route_decide(const RouteParams& p, float* L, float* PS, int* QS,
                                             int* slab_lds, int tok0) {
    const int tid = threadIdx.x;
    const int K = p.K, B = p.B, tok = tok0 + tid;
    const bool in_range = tok < p.N;
    const bool v = in_range && (p.valid == nullptr || p.valid[tok] != 0);
    float* row = L + tid * p.lstride;
    float* ps = PS + tid * (K + 1);
    int* qs = QS + tid * (K + 1);
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
            for (int c = 0; c < B; ++c) {
                const uint32_t uc = rank_key(u[c]);
                int rank = 0;
                for (int c2 = 0; c2 < B; ++c2) {
                    const uint32_t u2 = rank_key(u[c2]);
                    rank += (u2 > uc) || (u2 == uc && c2 < c);
                }
                if (rank < b) mask |= 1ull << c;
            }
        } else {
            mask = (b >= 64) ? ~0ull : ((1ull << b) - 1ull);
        }
        // Eq. residual-router-score: max-subtracted softmax, index-order sum.
        float* l = row + 1;
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
        for (int j = 0; j < K; ++j) {
            const float sj = l[j];
            const uint32_t kj = rank_key(sj);
            int rank = 0;
            for (int j2 = 0; j2 < K; ++j2) {
                const uint32_t k2 = rank_key(l[j2]);
                rank += (k2 > kj) || (k2 == kj && j2 < j);
            }
            ps[rank] = sj;
            qs[rank] = j + 1;
            p.eids[(size_t)tok * K + rank] = j + 1;
            p.wts[(size_t)tok * K + rank] = sj;
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
            p.eids[(size_t)tok * K + j] = -1;
            p.wts[(size_t)tok * K + j] = 0.f;
        }
    }
    if (p.bin_count == nullptr) return;

    // Pairs per (expert, key of the pair's block mask): one shared pair and
    // k residual pairs per valid token.
    const uint64_t full = (B == 64) ? ~0ull : ((1ull << B) - 1ull);
    const int kb = p.key_bits;
    if (v) {
        const uint64_t rmask = ~mask & full;
        const int ks = (int)(B > kb ? (mask >> (B - kb)) : mask);
        const int kr = (int)(B > kb ? (rmask >> (B - kb)) : rmask);
        atomicAdd(&p.bin_count[ks], 1);
        for (int i = 0; i < k; ++i) atomicAdd(&p.bin_count[(qs[i] << kb) + kr], 1);
    }
    // Rows per (expert, block): shared expert on I_shr, residual experts on I_res.
    const int lane = lane_id();
    for (int c = 0; c < B; ++c) {
        const uint64_t bits = ballot(v && ((mask >> c) & 1ull));
        if (lane == 0 && bits) atomicAdd(&slab_lds[c], __popcll(bits));
    }
    for (int e = 1; e <= K; ++e) {
        const bool has = v && ((sel >> (e - 1)) & 1ull);
        if (!ballot(has)) continue;
        for (int c = 0; c < B; ++c) {
            const uint64_t bits = ballot(has && !((mask >> c) & 1ull));
            if (lane == 0 && bits) atomicAdd(&slab_lds[e * B + c], __popcll(bits));
        }
    }
}

template <bool kBF16>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(RouteParams p) {
    extern __shared__ float lds_route[];
    float* L = lds_route;
    float* PS = L + kRouteTok * p.lstride;
    int* QS = reinterpret_cast<int*>(PS + kRouteTok * (p.K + 1));
    int* slab_lds = QS + kRouteTok * (p.K + 1);
    const int tok0 = blockIdx.x * kRouteTok;
    const int nslab = (p.K + 1) * p.B;
    if (p.slab_count)
        for (int i = threadIdx.x; i < nslab; i += blockDim.x) slab_lds[i] = 0;
    if (kBF16) route_logits_bf16(p, L, tok0);
    else route_logits_f32(p, L, tok0);
    __syncthreads();
    if (threadIdx.x < kRouteTok) route_decide(p, L, PS, QS, slab_lds, tok0);
    __syncthreads();
    if (p.slab_count)
        for (int i = threadIdx.x; i < nslab; i += blockDim.x)
            if (slab_lds[i]) atomicAdd(&p.slab_count[i], slab_lds[i]);
}

}  // namespace unifmoe
