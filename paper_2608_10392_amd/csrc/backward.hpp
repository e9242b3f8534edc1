// Backward pass of the layer (gradients of sum(dY * Y)), fp32 throughout.
//
// The discrete decisions (b, I_shr, q, k) are those of the forward and are
// held fixed; gradients flow through alpha (Eq. alpha) to W_shr and x,
// through the selected affinities p_i (the softmax of Eq.
// residual-router-score) to W_1..W_K and x, and through the expert FFNs of
// Eq. block-expert-output. The prototypes get none (they only enter TopK).
//
// A first, plain implementation (scalar fp32 FMA, no matrix cores):
//   bwd_pair      per (token, expert) pair: a = x K over the pair's active
//                 channels, act = GELU(a), E = act V, dcoef = dy . E,
//                 dE = w dy, dh = dE V^T, da = dh GELU'(a), dx_pair = da K^T
//   bwd_token     per token: dx = sum of its pairs' dx_pair, plus the router
//                 terms dz0 W_shr + sum_j dl_j W_j
//   bwd_wgrad     dW_up[e] = DA_e^T X_e and dW_down[e] = dE_e^T ACT_e over
//                 the pairs of expert e (tiled fp32 GEMMs, one 64 x 64 output
//                 tile per workgroup)
//   bwd_router    dW_router[j] = sum_t dz[t, j] x_t
#pragma once
#include "common.hpp"

namespace unifmoe {

struct BwdParams {
    int N, d, K, B, M, H;
    int alpha_adaptive;
    float tau, one_minus_2tau;
    const void* X;            // [N, d] layer format
    const void* dY;           // [N, d] layer format
    const void* Wup;          // [K+1, H, d]
    const void* Wdown;        // [K+1, d, H]
    const float* Wr;          // [K+1, d]
    const float* alpha;       // routing record
    const int* nres;
    const int* eids;          // [N, K]
    const float* wts;         // [N, K]
    const int* pair_token;    // forward pair tables (pairs grouped by expert)
    const int* pair_expert;
    const uint64_t* pair_mask;
    const int* pair_of;       // [N, K+1]
    const int* seg_off;       // [K+2] first pair of each expert segment
    const int* totals;        // [0]: pairs
    float* act;               // [pairs, H] GELU(a), zero on inactive channels
    float* da;                // [pairs, H] dL/da, zero on inactive channels
    float* dcoef;             // [pairs] dy . E_pair
    float* dxp;               // [pairs, d]
    float* dz;                // [N, K+1]: dz0, then dl_1..dl_K
    float* dX;                // [N, d]
    float* dWup;              // [K+1, H, d]
    float* dWdown;            // [K+1, d, H]
    float* dWr;               // [K+1, d]
};

template <bool BF16>
__device__ __forceinline__ float ld_val(const void* p, size_t i) {
    if constexpr (BF16) return bf2f(static_cast<const u16*>(p)[i]);
    else return static_cast<const float*>(p)[i];
}

// d GELU / da = Phi(a) + a phi(a).
__device__ __forceinline__ float gelu_grad_erf(float a) {
    return 0.5f * (1.0f + erff(a * 0.7071067811865475244f)) + a * 0.3989422804014327f * expf(-0.5f * a * a);
}

// Weight of pair (t, e): alpha for the shared expert, else the affinity p_i
// of the residual expert e = q_i.
__device__ __forceinline__ float pair_weight(const BwdParams& p, int t, int e) {
    if (e == 0) return p.alpha[t];
    const int k = p.nres[t];
    for (int i = 0; i < k; ++i)
        if (p.eids[(size_t)t * p.K + i] == e) return p.wts[(size_t)t * p.K + i];
    return 0.f;
}

__device__ __forceinline__ float block_sum(float v, float* red) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    float s = 0.f;
    for (int i = 0; i < nw; ++i) s += red[i];
    return s;
}

// One workgroup per pair (grid-stride). LDS: x, dE (d floats each), act and
// da (H floats each), 16 floats for reductions.
template <bool BF16>
__global__ __launch_bounds__(256) void bwd_pair_kernel(BwdParams p) {
    extern __shared__ float lds_b[];
    float* xs = lds_b;
    float* dEs = xs + p.d;
    float* acts = dEs + p.d;
    float* das = acts + p.H;
    float* red = das + p.H;
    const int P = p.totals[0];
    for (int pr = blockIdx.x; pr < P; pr += gridDim.x) {
        const int t = p.pair_token[pr], e = p.pair_expert[pr];
        const uint64_t mask = p.pair_mask[pr];
        const float w = pair_weight(p, t, e);
        __syncthreads();
        for (int n = threadIdx.x; n < p.d; n += blockDim.x) {
            xs[n] = ld_val<BF16>(p.X, (size_t)t * p.d + n);
            dEs[n] = w * ld_val<BF16>(p.dY, (size_t)t * p.d + n);
        }
        __syncthreads();
        // Channels: a, act, dh, da.
        for (int h = threadIdx.x; h < p.H; h += blockDim.x) {
            float act = 0.f, dah = 0.f;
            if ((mask >> (h / p.M)) & 1ull) {
                const size_t urow = ((size_t)e * p.H + h) * p.d;
                float a = 0.f;
                for (int n = 0; n < p.d; ++n) a = fmaf(ld_val<BF16>(p.Wup, urow + n), xs[n], a);
                act = gelu_erf(a);
                float dh = 0.f;
                const size_t dbase = (size_t)e * p.d * p.H + h;
                for (int n = 0; n < p.d; ++n) dh = fmaf(ld_val<BF16>(p.Wdown, dbase + (size_t)n * p.H), dEs[n], dh);
                dah = dh * gelu_grad_erf(a);
            }
            acts[h] = act;
            das[h] = dah;
            p.act[(size_t)pr * p.H + h] = act;
            p.da[(size_t)pr * p.H + h] = dah;
        }
        __syncthreads();
        // Outputs: E (for dcoef) and dx_pair.
        float dc = 0.f;
        for (int n = threadIdx.x; n < p.d; n += blockDim.x) {
            const size_t drow = ((size_t)e * p.d + n) * p.H;
            float E = 0.f, dx = 0.f;
            for (int c = 0; c < p.B; ++c) {
                if (!((mask >> c) & 1ull)) continue;
                for (int h = c * p.M; h < (c + 1) * p.M; ++h) {
                    E = fmaf(ld_val<BF16>(p.Wdown, drow + h), acts[h], E);
                    dx = fmaf(ld_val<BF16>(p.Wup, ((size_t)e * p.H + h) * p.d + n), das[h], dx);
                }
            }
            dc = fmaf(ld_val<BF16>(p.dY, (size_t)t * p.d + n), E, dc);
            p.dxp[(size_t)pr * p.d + n] = dx;
        }
        dc = block_sum(dc, red);
        if (threadIdx.x == 0) p.dcoef[pr] = dc;
    }
}

// One wave per token: router terms and the sum of the token's pairs.
__global__ __launch_bounds__(256) void bwd_token_kernel(BwdParams p) {
    const int t = blockIdx.x * (blockDim.x >> 6) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (t >= p.N) return;
    const int lane = lane_id();
    const int k = p.nres[t];
    const int* of = p.pair_of + (size_t)t * (p.K + 1);
    float* dz = p.dz + (size_t)t * (p.K + 1);
    if (k == 0) {   // padded token
        for (int j = lane; j <= p.K; j += kWave) dz[j] = 0.f;
        for (int n = lane; n < p.d; n += kWave) p.dX[(size_t)t * p.d + n] = 0.f;
        return;
    }
    // alpha = tau + (1 - 2 tau) sigma(z0): dz0 = dcoef_shr (1 - 2 tau) sigma (1 - sigma),
    // sigma recovered from alpha.
    float dz0 = 0.f;
    if (p.alpha_adaptive) {
        const float sg = (p.alpha[t] - p.tau) / p.one_minus_2tau;
        dz0 = p.dcoef[of[0]] * p.one_minus_2tau * sg * (1.f - sg);
    }
    // p_i = s_{q_i}; dl_{q_i} = p_i (dp_{q_i} - sum_m p_m dp_{q_m}), dp nonzero for i < k.
    float sdp = 0.f;
    for (int i = 0; i < k; ++i) sdp = fmaf(p.wts[(size_t)t * p.K + i], p.dcoef[of[1 + i]], sdp);
    // dz (for the router's weight gradient, a later kernel) and dX: every
    // lane recomputes the K values dl_j it needs rather than reading dz back.
    if (lane == 0) dz[0] = dz0;
    for (int i = lane; i < p.K; i += kWave) {
        const float pi = p.wts[(size_t)t * p.K + i];
        const float dpi = (i < k) ? p.dcoef[of[1 + i]] : 0.f;
        dz[p.eids[(size_t)t * p.K + i]] = pi * (dpi - sdp);
    }
    for (int n = lane; n < p.d; n += kWave) {
        float v = 0.f;
        for (int i = 0; i <= k; ++i) v += p.dxp[(size_t)of[i] * p.d + n];
        v = fmaf(dz0, p.Wr[n], v);
        for (int i = 0; i < p.K; ++i) {
            const float pi = p.wts[(size_t)t * p.K + i];
            const float dpi = (i < k) ? p.dcoef[of[1 + i]] : 0.f;
            v = fmaf(pi * (dpi - sdp), p.Wr[(size_t)p.eids[(size_t)t * p.K + i] * p.d + n], v);
        }
        p.dX[(size_t)t * p.d + n] = v;
    }
}

// dW_router[j][n] = sum_t dz[t][j] x_t[n]: one thread per (j, n).
template <bool BF16>
__global__ __launch_bounds__(256) void bwd_router_kernel(BwdParams p) {
    const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (item >= (size_t)(p.K + 1) * p.d) return;
    const int j = (int)(item / p.d), n = (int)(item - (size_t)j * p.d);
    float s = 0.f;
    for (int t = 0; t < p.N; ++t) s = fmaf(p.dz[(size_t)t * (p.K + 1) + j], ld_val<BF16>(p.X, (size_t)t * p.d + n), s);
    p.dWr[item] = s;
}

// Weight gradients of expert e as two fp32 GEMMs over its pair segment:
//   dW_up[e][h][n]   = sum_pr da[pr][h] x_{tok(pr)}[n]
//   dW_down[e][n][h] = sum_pr w_pr dy_{tok(pr)}[n] act[pr][h]
// blockIdx.z = e, blockIdx.y picks the product (0: up, 1: down); one 64 x 64
// output tile per workgroup (rows: h for up, n for down), 16 pairs per LDS
// step, 4 x 4 outputs per thread.
template <bool BF16>
__global__ __launch_bounds__(256) void bwd_wgrad_kernel(BwdParams p, int tiles_h, int tiles_d) {
    __shared__ float Ls[16][64 + 1];   // pair x output-row operand
    __shared__ float Rs[16][64 + 1];   // pair x output-column operand
    const int e = blockIdx.z, up = blockIdx.y == 0;
    const int rows = up ? p.H : p.d, cols = up ? p.d : p.H;
    const int tr = up ? tiles_h : tiles_d, tc = up ? tiles_d : tiles_h;
    const int tile = blockIdx.x;
    if (tile >= tr * tc) return;
    const int r0 = (tile / tc) * 64, c0 = (tile % tc) * 64;
    const int p0 = p.seg_off[e], p1 = p.seg_off[e + 1];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    float acc[4][4] = {};
    for (int q0 = p0; q0 < p1; q0 += 16) {
        // Stage 16 pairs x 64 rows and 16 pairs x 64 columns.
        for (int i = threadIdx.x; i < 16 * 64; i += blockDim.x) {
            const int pi = i / 64, x = i % 64, pr = q0 + pi;
            float lv = 0.f, rv = 0.f;
            if (pr < p1) {
                const int t = p.pair_token[pr];
                if (up) {
                    if (r0 + x < rows) lv = p.da[(size_t)pr * p.H + r0 + x];
                    if (c0 + x < cols) rv = ld_val<BF16>(p.X, (size_t)t * p.d + c0 + x);
                } else {
                    const float w = pair_weight(p, t, e);
                    if (r0 + x < rows) lv = w * ld_val<BF16>(p.dY, (size_t)t * p.d + r0 + x);
                    if (c0 + x < cols) rv = p.act[(size_t)pr * p.H + c0 + x];
                }
            }
            Ls[pi][x] = lv;
            Rs[pi][x] = rv;
        }
        __syncthreads();
#pragma unroll 4
        for (int pi = 0; pi < 16; ++pi) {
            float l[4], r[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                l[u] = Ls[pi][ty * 4 + u];
                r[u] = Rs[pi][tx * 4 + u];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(l[u], r[v], acc[u][v]);
        }
        __syncthreads();
    }
    float* out = up ? p.dWup + (size_t)e * p.H * p.d : p.dWdown + (size_t)e * p.d * p.H;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int r = r0 + ty * 4 + u;
        if (r >= rows) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int c = c0 + tx * 4 + v;
            if (c < cols) out[(size_t)r * cols + c] = acc[u][v];
        }
    }
}

}  // namespace unifmoe
