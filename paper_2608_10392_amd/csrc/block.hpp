// The transformer block around the layer: LayerNorm of the FFN input
// (pre-LN) and the block's merge (Eq. output plus the b2 shares, the
// residual add and, post-LN, the LayerNorm of the sum).
//
// LayerNorm: LN(v) = (v - mean) / sqrt(var + eps) * gamma + beta, biased
// variance over the d features. Statistics and the normalisation run in
// fp64 (sums of d terms; the result then differs from the exact value by a
// few fp64 ulps, so rounding it to the layer's format almost never lands on
// the other side of a rounding midpoint). One wave per row; every lane ends
// a butterfly reduction with the same (commutative) sums.
#pragma once
#include "common.hpp"

namespace unifmoe {

// Both kernels take one row per wave and blockDim.x / 64 rows per workgroup.

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

__device__ __forceinline__ float load_elem(const void* row, int j, bool bf16) {
    return bf16 ? bf2f(static_cast<const u16*>(row)[j]) : static_cast<const float*>(row)[j];
}

__device__ __forceinline__ void store_elem(void* row, int j, double v, bool bf16) {
    if (bf16) static_cast<u16*>(row)[j] = f64_to_bf16(v);
    else static_cast<float*>(row)[j] = (float)v;
}

// mean and 1 / sqrt(var + eps) of a row read through get(j) (fp64).
template <typename G>
__device__ __forceinline__ void row_moments(G get, int d, double eps, double& mu, double& rstd) {
    const int lane = lane_id();
    double s = 0.0;
    for (int j = lane; j < d; j += kWave) s += (double)get(j);
    mu = wave_sum_f64(s) / d;
    double q = 0.0;
    for (int j = lane; j < d; j += kWave) {
        const double c = (double)get(j) - mu;
        q = fma(c, c, q);
    }
    rstd = 1.0 / sqrt(wave_sum_f64(q) / d + eps);
}

// Pre-LN: Xn = LN(X), one wave per row (the row is re-read from cache by
// each pass).
template <bool BF16>
__global__ __launch_bounds__(256) void layernorm_rows_kernel(LayerNormParams p) {
    const int t = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    if (t >= p.N) return;
    const size_t esz = BF16 ? 2 : 4;
    const char* xr = static_cast<const char*>(p.X) + (size_t)t * p.d * esz;
    char* yr = static_cast<char*>(p.Xn) + (size_t)t * p.d * esz;
    auto get = [&](int j) { return load_elem(xr, j, BF16); };
    double mu, rstd;
    row_moments(get, p.d, p.eps, mu, rstd);
    for (int j = lane_id(); j < p.d; j += kWave) {
        const double v = ((double)get(j) - mu) * rstd * (double)p.gamma[j] + (double)p.beta[j];
        store_elem(yr, j, v, BF16);
    }
}

struct BlockCombineParams {
    int N, d, K, B;
    const void* part;       // per-pair expert rows (layer format)
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
};

// One wave per token. z_j = alpha E_shr^S + sum_{i <= k} p_i E_{q_i}^R
// (the expert rows in the layer's fixed order, fp32), then the b2 shares
// alpha (b/B) b2_shr + sum_i p_i ((B-b)/B) b2_{q_i}, then x_j. Post-LN keeps
// z in LDS (d floats per wave) for the LayerNorm.
template <bool BF16>
__global__ __launch_bounds__(256) void combine_block_kernel(BlockCombineParams c) {
    extern __shared__ float zrow_all[];
    const int w = threadIdx.x >> 6;
    const int t = blockIdx.x * (blockDim.x >> 6) + w;
    if (t >= c.N) return;
    float* zrow = zrow_all + (size_t)w * c.d;
    const int lane = lane_id();
    const int k = c.nres[t];
    const int b = c.nsh[t];
    const float a = c.alpha[t];
    const float share_s = (float)b / (float)c.B, share_r = (float)(c.B - b) / (float)c.B;
    const int* of = c.pair_of + (size_t)t * (c.K + 1);
    const int* q = c.eids + (size_t)t * c.K;
    const float* wt = c.wts + (size_t)t * c.K;
    const size_t esz = BF16 ? 2 : 4;
    const char* xr = c.X ? static_cast<const char*>(c.X) + (size_t)t * c.d * esz : nullptr;
    char* yr = static_cast<char*>(c.Y) + (size_t)t * c.d * esz;
    const char* part = static_cast<const char*>(c.part);
    double s = 0.0;
    for (int j = lane; j < c.d; j += kWave) {
        float z = 0.f;
        if (k > 0) {
            for (int i = 0; i <= k; ++i) {
                const float wi = (i == 0) ? a : wt[i - 1];
                z = fmaf(wi, load_elem(part + (size_t)of[i] * c.d * esz, j, BF16), z);
            }
            if (c.b_down != nullptr) {
                z = fmaf(a * share_s, c.b_down[j], z);
                for (int i = 1; i <= k; ++i) z = fmaf(wt[i - 1] * share_r, c.b_down[(size_t)q[i - 1] * c.d + j], z);
            }
        }
        if (xr != nullptr) z += load_elem(xr, j, BF16);
        if (c.post) {
            zrow[j] = z;
            s += (double)z;
        } else {
            store_elem(yr, j, (double)z, BF16);
        }
    }
    if (!c.post) return;
    // Each lane reads back only the entries it wrote (j = lane + 64 i), so
    // no barrier is needed between the passes.
    const double mu = wave_sum_f64(s) / c.d;
    double sq = 0.0;
    for (int j = lane; j < c.d; j += kWave) {
        const double e = (double)zrow[j] - mu;
        sq = fma(e, e, sq);
    }
    const double rstd = 1.0 / sqrt(wave_sum_f64(sq) / c.d + c.eps);
    for (int j = lane; j < c.d; j += kWave) {
        const double v = ((double)zrow[j] - mu) * rstd * (double)c.gamma[j] + (double)c.beta[j];
        store_elem(yr, j, v, BF16);
    }
}

}  // namespace unifmoe
