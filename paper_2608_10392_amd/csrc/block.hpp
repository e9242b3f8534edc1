// The transformer block around the layer: LayerNorm of the FFN input
// (pre-LN) and the block's merge (Eq. output plus the b2 shares, the
// residual add and, post-LN, the LayerNorm of the sum).
//
// LayerNorm: LN(v) = (v - mean) / sqrt(var + eps) * gamma + beta, biased
// variance over the d features. Statistics and the normalisation run in
// fp64 (sums of d terms; the result then differs from the exact value by a
// few fp64 ulps, so rounding it to the layer's format almost never lands on
// the other side of a rounding midpoint). Row sums are butterfly
// reductions over the lanes of a row, after which every one of those lanes
// holds the same (commutative) sums.
#pragma once
#include "common.hpp"

namespace unifmoe {

// The post-LN merge takes one row per wave and blockDim.x / 64 rows per
// workgroup; the LayerNorm pass takes LPR lanes per row.

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// fp64 -> bf16, round to nearest even, via round-to-odd fp32: the fp32 value
// truncated toward zero, with its last bit set when inexact; rounding that
// to 8 significant bits equals rounding the fp64 value directly (the fp32
// format has at least two more bits), in the normal range.
__device__ __forceinline__ u16 f64_to_bf16(double v) {
    float f = __double2float_rz(v);
    if ((double)f != v) f = __uint_as_float(__float_as_uint(f) | 1u);
    return f2bf(f);
}

struct LayerNormParams {
    int N, d;
    const void* X;      // [N, d] layer format
    void* Xn;           // [N, d] layer format
    const float* gamma;
    const float* beta;
    double eps;
};

// Rows are walked in chunks: 8 bf16 (one 16-byte access) or one fp32
// element; lane l takes chunks l, l + 64, ...
template <bool BF16>
struct Chunk {
    static constexpr int E = BF16 ? 8 : 1;
    float v[E];
    __device__ __forceinline__ void load(const void* row, int ch) {
        if constexpr (BF16) {
            const u32x4 q = ld16(static_cast<const u16*>(row) + ch * 8);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[2 * i] = __uint_as_float(q[i] << 16);
                v[2 * i + 1] = __uint_as_float(q[i] & 0xffff0000u);
            }
        } else {
            v[0] = static_cast<const float*>(row)[ch];
        }
    }
};

template <bool BF16>
__device__ __forceinline__ void store_chunk(void* row, int ch, const double (&y)[Chunk<BF16>::E]) {
    if constexpr (BF16) {
        u32x4 q;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            q[i] = (uint32_t)f64_to_bf16(y[2 * i]) | ((uint32_t)f64_to_bf16(y[2 * i + 1]) << 16);
        st16(static_cast<u16*>(row) + ch * 8, q);
    } else {
        static_cast<float*>(row)[ch] = (float)y[0];
    }
}

// Sum over the LPR consecutive lanes that share a row (LPR a power of two
// <= 64); every lane of the group ends with the same sum.
template <int LPR>
__device__ __forceinline__ double group_sum_f64(double v) {
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// Pre-LN: Xn = LN(X), LPR lanes per row (several rows per wave, so each
// wave keeps more loads in flight). Rows of at most LPR MAXC chunks stay in
// registers (one read); longer rows are re-read from cache by each of the
// three passes (mean, variance, output).
template <bool BF16, int MAXC, int LPR>
__global__ __launch_bounds__(256) void layernorm_rows_kernel(LayerNormParams p) {
    using C = Chunk<BF16>;
    const int t = (int)((blockIdx.x * blockDim.x + threadIdx.x) / LPR);
    if (t >= p.N) return;
    const int sub = threadIdx.x % LPR, nch = p.d / C::E;
    const size_t esz = BF16 ? 2 : 4;
    const char* xr = static_cast<const char*>(p.X) + (size_t)t * p.d * esz;
    char* yr = static_cast<char*>(p.Xn) + (size_t)t * p.d * esz;
    const bool cached = nch <= LPR * MAXC;
    C cache[MAXC];
    if (cached) {
#pragma unroll
        for (int i = 0; i < MAXC; ++i)
            if (sub + LPR * i < nch) cache[i].load(xr, sub + LPR * i);
    }
    // Chunk ch = sub + LPR i of the row, from registers or from memory.
    auto chunk = [&](int i, int ch) {
        C c;
        if (cached) {
#pragma unroll
            for (int j = 0; j < MAXC; ++j)
                if (j == i) c = cache[j];
        } else {
            c.load(xr, ch);
        }
        return c;
    };
    double s = 0.0;
    for (int i = 0, ch = sub; ch < nch; ++i, ch += LPR) {
        const C c = chunk(i, ch);
#pragma unroll
        for (int e = 0; e < C::E; ++e) s += (double)c.v[e];
    }
    const double mu = group_sum_f64<LPR>(s) / p.d;
    double q = 0.0;
    for (int i = 0, ch = sub; ch < nch; ++i, ch += LPR) {
        const C c = chunk(i, ch);
#pragma unroll
        for (int e = 0; e < C::E; ++e) {
            const double u = (double)c.v[e] - mu;
            q = fma(u, u, q);
        }
    }
    const double rstd = 1.0 / sqrt(group_sum_f64<LPR>(q) / p.d + p.eps);
    for (int i = 0, ch = sub; ch < nch; ++i, ch += LPR) {
        const C c = chunk(i, ch);
        double y[C::E];
#pragma unroll
        for (int e = 0; e < C::E; ++e) {
            const int j = ch * C::E + e;
            y[e] = ((double)c.v[e] - mu) * rstd * (double)p.gamma[j] + (double)p.beta[j];
        }
        store_chunk<BF16>(yr, ch, y);
    }
}

struct BlockCombineParams {
    int N, d, K, B;
    int nsplit;             // row buffers per pair (bf16: the down-projection's parts), summed in order
    size_t split_stride;    // floats between them
    const void* part;       // per-pair expert rows (fp32)
    const int* pair_of;     // [N, K+1] pair of (token, i-th pathway)
    const float* alpha;
    const int* nsh;         // b
    const int* nres;        // k
    const int* eids;        // [N, K] q_1..q_K
    const float* wts;       // [N, K] p_1..p_K
    const float* b_down;    // [K+1, d] or null
    const void* X;          // block input (residual), null: no residual add
    int post;               // nonzero: LayerNorm of the sum
    const float* gamma;
    const float* beta;
    double eps;
    void* Y;
    const int* totals;      // totals[5] != 0: the routing overflowed the pair capacity (Y = 0)
};

constexpr int kBlockCombineBatch = 4;

// z over one chunk of token t's row: alpha E_shr^S + sum_{i <= k} p_i
// E_{q_i}^R (the expert rows in the layer's fixed order, fp32, loaded in
// batches), then the b2 shares alpha (b/B) b2_shr + sum_i p_i ((B-b)/B)
// b2_{q_i}, then x.
template <bool BF16>
__device__ __forceinline__ void block_chunk_sum(const BlockCombineParams& c, int t, int ch,
                                                float (&z)[Chunk<BF16>::E]) {
    using C = Chunk<BF16>;
    constexpr int E = C::E;
    const int k = c.nres[t];
    const float a = c.alpha[t];
    const int* of = c.pair_of + (size_t)t * (c.K + 1);
    const float* wt = c.wts + (size_t)t * c.K;
    const size_t esz = BF16 ? 2 : 4;
    const float* part = static_cast<const float*>(c.part);
#pragma unroll
    for (int e = 0; e < E; ++e) z[e] = 0.f;
    for (int i0 = 0; i0 <= k && k > 0; i0 += kBlockCombineBatch) {
        float r[kBlockCombineBatch][E];
#pragma unroll
        for (int u = 0; u < kBlockCombineBatch; ++u) {
            if (i0 + u <= k) {
                const float* row = part + (size_t)of[i0 + u] * c.d + ch * E;
                if constexpr (BF16) {
#pragma unroll
                    for (int h = 0; h < E / 4; ++h) {
                        f32x4 q = *reinterpret_cast<const f32x4*>(row + 4 * h);
                        for (int sp = 1; sp < c.nsplit; ++sp)
                            q += *reinterpret_cast<const f32x4*>(row + sp * c.split_stride + 4 * h);
#pragma unroll
                        for (int e = 0; e < 4; ++e) r[u][4 * h + e] = q[e];
                    }
                } else {
                    r[u][0] = row[0];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kBlockCombineBatch; ++u) {
            if (i0 + u <= k) {
                const float wi = (i0 + u == 0) ? a : wt[i0 + u - 1];
#pragma unroll
                for (int e = 0; e < E; ++e) z[e] = fmaf(wi, r[u][e], z[e]);
            }
        }
    }
    if (c.b_down != nullptr && k > 0) {
        const int b = c.nsh[t];
        const float share_s = (float)b / (float)c.B, share_r = (float)(c.B - b) / (float)c.B;
        const int* q = c.eids + (size_t)t * c.K;
        // b2 rows: E consecutive floats (16-byte aligned for bf16 layers).
        auto add_b2 = [&](const float* row, float f) {
            if constexpr (BF16) {
#pragma unroll
                for (int h = 0; h < E / 4; ++h) {
                    const f32x4 b4 = *reinterpret_cast<const f32x4*>(row + 4 * h);
#pragma unroll
                    for (int e = 0; e < 4; ++e) z[4 * h + e] = fmaf(f, b4[e], z[4 * h + e]);
                }
            } else {
                z[0] = fmaf(f, row[0], z[0]);
            }
        };
        add_b2(c.b_down + ch * E, a * share_s);
        for (int i = 1; i <= k; ++i) add_b2(c.b_down + (size_t)q[i - 1] * c.d + ch * E, wt[i - 1] * share_r);
    }
    if (c.X != nullptr) {
        C x;
        x.load(static_cast<const char*>(c.X) + (size_t)t * c.d * esz, ch);
#pragma unroll
        for (int e = 0; e < E; ++e) z[e] += x.v[e];
    }
}

// No post-LN: one thread per chunk of the whole output (the layer's
// combine layout).
template <bool BF16>
__global__ __launch_bounds__(256) void combine_block_flat_kernel(BlockCombineParams c) {
    constexpr int E = Chunk<BF16>::E;
    const int nch = c.d / E;
    const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (item >= (size_t)c.N * nch) return;
    const int t = (int)(item / nch), ch = (int)(item - (size_t)t * nch);
    float z[E];
    if (ld_uniform(c.totals + 5) != 0) {
        // past the pair capacity no expert row exists: Y = 0
#pragma unroll
        for (int e = 0; e < E; ++e) z[e] = 0.f;
    } else {
        block_chunk_sum<BF16>(c, t, ch, z);
    }
    // One rounding from fp32 (what f64_to_bf16 gives for an fp32 value).
    if constexpr (BF16) {
        u32x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (uint32_t)f2bf(z[2 * i]) | ((uint32_t)f2bf(z[2 * i + 1]) << 16);
        st16(static_cast<u16*>(c.Y) + (size_t)t * c.d + ch * 8, o);
    } else {
        static_cast<float*>(c.Y)[(size_t)t * c.d + ch] = z[0];
    }
}

// Post-LN: one wave per token; z stays in LDS (d floats per wave; each lane
// reads back only what it wrote) for the LayerNorm.
template <bool BF16>
__global__ __launch_bounds__(256) void combine_block_post_kernel(BlockCombineParams c) {
    constexpr int E = Chunk<BF16>::E;
    extern __shared__ float zrow_all[];
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int t = blockIdx.x * (blockDim.x >> 6) + w;
    if (t >= c.N) return;
    float* zrow = zrow_all + (size_t)w * c.d;
    const int lane = lane_id(), nch = c.d / E;
    char* yr = static_cast<char*>(c.Y) + (size_t)t * c.d * (BF16 ? 2 : 4);
    if (ld_uniform(c.totals + 5) != 0) {
        // past the pair capacity no expert row exists: Y = 0
        double y0[E];
#pragma unroll
        for (int e = 0; e < E; ++e) y0[e] = 0.0;
        for (int ch = lane; ch < nch; ch += kWave) store_chunk<BF16>(yr, ch, y0);
        return;
    }
    double s = 0.0;
    for (int ch = lane; ch < nch; ch += kWave) {
        float z[E];
        block_chunk_sum<BF16>(c, t, ch, z);
#pragma unroll
        for (int e = 0; e < E; ++e) {
            zrow[ch * E + e] = z[e];
            s += (double)z[e];
        }
    }
    const double mu = wave_sum_f64(s) / c.d;
    double sq = 0.0;
    for (int ch = lane; ch < nch; ch += kWave) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const double u = (double)zrow[ch * E + e] - mu;
            sq = fma(u, u, sq);
        }
    }
    const double rstd = 1.0 / sqrt(wave_sum_f64(sq) / c.d + c.eps);
    for (int ch = lane; ch < nch; ch += kWave) {
        double y[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int j = ch * E + e;
            y[e] = ((double)zrow[j] - mu) * rstd * (double)c.gamma[j] + (double)c.beta[j];
        }
        store_chunk<BF16>(yr, ch, y);
    }
}

}  // namespace unifmoe
