// Backward pass of the layer (gradients of sum(dY * Y)).
//
// The discrete decisions (b, I_shr, q, k) are those of the forward and are
// held fixed; gradients flow through alpha (Eq. alpha) to W_shr and x,
// through the selected affinities p_i (the softmax of Eq.
// residual-router-score) to W_1..W_K and x, and through the expert FFNs of
// Eq. block-expert-output. The prototypes get none (they only enter TopK).
//
// bf16 layers run on the matrix cores (the up and down engines of
// ffn_bf16.hpp with backward epilogues, and wgrad.hpp); the kernels here
// serve them for the per-pair and per-token scalars (bwd_weight_kernel,
// bwd_dcoef_sum_kernel, bwd_token_kernel, the router kernels).
//
// fp32 layers run on the vector units (fp32 FMA) as tiled fp32 GEMMs over
// each expert's segment of pairs (rows gathered by token; dense over the H
// channels, masked to the pair's blocks):
//   bwd_seg<0>    a = x K^T; act = GELU(a), gp = GELU'(a) on active channels
//   bwd_seg<1>    E = act V^T                        (per-pair expert output)
//   bwd_dcoef     dcoef = dy . E                     (d loss / d pair weight)
//   bwd_seg<2>    dh = dE V, dE = w dy; da = dh gp
//   bwd_seg<3>    dx_pair = da K
//   bwd_token     per token: dx = sum of its pairs' dx_pair, plus the router
//                 terms dz0 W_shr + sum_j dl_j W_j
//   bwd_wgrad     dW_up[e] = DA_e^T X_e and dW_down[e] = dE_e^T ACT_e over
//                 the pairs of expert e
//   bwd_router    dW_router[j] = sum_t dz[t, j] x_t (token slices, then
//                 their sum)
#pragma once
#include <type_traits>

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
    float* da;                // [pairs, H] GELU'(a), then dL/da; zero on inactive channels
    float* dcoef;             // [pairs] dy . E_pair
    float* pw;                // [pairs] pair weight (alpha or p_i)
    float* dxp;               // [pairs, d] E_pair, then dx_pair
    float* dz;                // [N, K+1]: dz0, then dl_1..dl_K
    float* rpart;             // [kRouterChunks, K+1, d] partial router gradients
    float* dX;                // [N, d]
    float* dWup;              // [K+1, H, d]
    float* dWdown;            // [K+1, d, H]
    float* dWr;               // [K+1, d]
};

__device__ __forceinline__ float ld_f32(const void* p, size_t i) { return static_cast<const float*>(p)[i]; }


// Blocks (bit c) that channels [h0, h1) touch, h0 < h1.
__device__ __forceinline__ uint64_t channel_blocks(int h0, int h1, int M) {
    const int b0 = h0 / M, b1 = (h1 - 1) / M;
    const uint64_t hi = (b1 >= 63) ? ~0ull : ((1ull << (b1 + 1)) - 1);
    return hi & ~((1ull << b0) - 1);
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

// Pair weights: alpha for the shared expert, p_i for residual expert q_i.
__global__ __launch_bounds__(256) void bwd_weight_kernel(BwdParams p) {
    const int P = p.totals[0];
    for (int pr = blockIdx.x * blockDim.x + threadIdx.x; pr < P; pr += gridDim.x * blockDim.x)
        p.pw[pr] = pair_weight(p, p.pair_token[pr], p.pair_expert[pr]);
}

// dcoef[pr] = dy_{tok(pr)} . E_pr from the partial sums the bf16 path's
// second up-projection leaves per (pair, block, column half): summed over
// the blocks of the pair's mask in increasing order (a pair with no block
// gets 0).
__global__ __launch_bounds__(256) void bwd_dcoef_sum_kernel(BwdParams p, const float* __restrict__ dcp) {
    const int P = p.totals[0];
    for (int pr = blockIdx.x * blockDim.x + threadIdx.x; pr < P; pr += gridDim.x * blockDim.x) {
        uint64_t m = p.pair_mask[pr];
        float s = 0.f;
        while (m) {
            const float* q = dcp + ((size_t)pr * p.B + __builtin_ctzll(m)) * 2;
            s += q[0] + q[1];
            m &= m - 1;
        }
        p.dcoef[pr] = s;
    }
}

// dcoef[pr] = dy_{tok(pr)} . E_pr, one wave per pair (fp32 path).
__global__ __launch_bounds__(256) void bwd_dcoef_kernel(BwdParams p) {
    const int pr = blockIdx.x * (blockDim.x >> 6) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (pr >= p.totals[0]) return;
    const int t = p.pair_token[pr];
    float s = 0.f;
    for (int n = lane_id(); n < p.d; n += kWave)
        s = fmaf(ld_f32(p.dY, (size_t)t * p.d + n), p.dxp[(size_t)pr * p.d + n], s);
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane_id() == 0) p.dcoef[pr] = s;
}

// Output tile of the backward GEMMs: kBT x kBT per workgroup of 256
// threads, kBU x kBU per thread, 16 k per LDS step.
constexpr int kBT = 128, kBU = kBT / 16;

// C[pr][col] = sum_k L(pr, k) R(k, col) over the pairs of expert e =
// blockIdx.z, one kBT x kBT tile per workgroup (blockIdx.y: pair tile,
// blockIdx.x: column tile; tiles past the segment exit).
//   MODE 0: L = x (k over d), R = K^T (col = channel h)      -> act, gp
//   MODE 1: L = act (k over H), R = V^T (col = output n)      -> E
//   MODE 2: L = w dy (k over d), R = V (col = channel h)      -> da = dh gp
//   MODE 3: L = da (k over H), R = K (col = output n)         -> dx_pair
template <int MODE>
__global__ __launch_bounds__(256) void bwd_seg_kernel(BwdParams p) {
    __shared__ float Ls[16][kBT + 1];
    __shared__ float Rs[16][kBT + 1];
    constexpr bool CH = (MODE == 0 || MODE == 2);   // columns are channels
    constexpr bool KD = (MODE == 0 || MODE == 2);   // contraction over d
    const int e = blockIdx.z;
    const int p0 = p.seg_off[e], p1 = p.seg_off[e + 1];
    const int r0 = p0 + (int)blockIdx.y * kBT;
    const int cols = CH ? p.H : p.d, kdim = KD ? p.d : p.H;
    const int c0 = (int)blockIdx.x * kBT;
    if (r0 >= p1 || c0 >= cols) return;
    const size_t wu = (size_t)e * p.H * p.d, wd = (size_t)e * p.d * p.H;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    // Union of the block masks of the tile's pairs. Pairs are sorted by mask
    // key, so a tile's pairs mostly agree on a block, and a block none of
    // them runs contributes exact zeros: channel tiles of such blocks are
    // skipped (MODE 0 writes zeros), and so are k steps inside them.
    __shared__ uint64_t un_w[kBT / 64];
    if (threadIdx.x < kBT) {
        const int pr = r0 + threadIdx.x;
        uint64_t m = pr < p1 ? p.pair_mask[pr] : 0ull;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) m |= shfl_xor64(m, o);
        if (lane_id() == 0) un_w[threadIdx.x >> 6] = m;
    }
    __syncthreads();
    uint64_t un = 0;
#pragma unroll
    for (int w = 0; w < kBT / 64; ++w) un |= un_w[w];
    if constexpr (CH) {
        if ((un & channel_blocks(c0, min(c0 + kBT, cols), p.M)) == 0) {
            if constexpr (MODE == 0) {
                for (int i = threadIdx.x; i < kBT * kBT; i += blockDim.x) {
                    const int pr = r0 + i / kBT, col = c0 + i % kBT;
                    if (pr < p1 && col < cols) {
                        p.act[(size_t)pr * p.H + col] = 0.f;
                        p.da[(size_t)pr * p.H + col] = 0.f;
                    }
                }
            }
            return;
        }
    }
    float acc[kBU][kBU] = {};
    for (int k0 = 0; k0 < kdim; k0 += 16) {
        if constexpr (!KD) {
            // skip a 16-channel step only if no pair of the tile runs any
            // block it touches (with M % 16 != 0 a step spans two blocks)
            if ((un & channel_blocks(k0, min(k0 + 16, kdim), p.M)) == 0) continue;
        }
        for (int i = threadIdx.x; i < 16 * kBT; i += blockDim.x) {
            // L: kBT pair rows x 16 k, consecutive threads along k.
            {
                const int r = i / 16, kk = i % 16, pr = r0 + r, k = k0 + kk;
                float v = 0.f;
                if (pr < p1 && k < kdim) {
                    if constexpr (MODE == 0) v = ld_f32(p.X, (size_t)p.pair_token[pr] * p.d + k);
                    else if constexpr (MODE == 1) v = p.act[(size_t)pr * p.H + k];
                    else if constexpr (MODE == 2) v = p.pw[pr] * ld_f32(p.dY, (size_t)p.pair_token[pr] * p.d + k);
                    else v = p.da[(size_t)pr * p.H + k];
                }
                Ls[kk][r] = v;
            }
            // R: 16 k x kBT columns, consecutive threads along the weight's
            // contiguous index.
            {
                float v = 0.f;
                if constexpr (MODE == 0 || MODE == 1) {
                    const int c = i / 16, kk = i % 16, col = c0 + c, k = k0 + kk;
                    if (col < cols && k < kdim)
                        v = MODE == 0 ? ld_f32(p.Wup, wu + (size_t)col * p.d + k)       // K_e[h = col][n = k]
                                      : ld_f32(p.Wdown, wd + (size_t)col * p.H + k);    // V_e[n = col][h = k]
                    Rs[kk][c] = v;
                } else {
                    const int kk = i / kBT, c = i % kBT, col = c0 + c, k = k0 + kk;
                    if (col < cols && k < kdim)
                        v = MODE == 2 ? ld_f32(p.Wdown, wd + (size_t)k * p.H + col)     // V_e[n = k][h = col]
                                      : ld_f32(p.Wup, wu + (size_t)k * p.d + col);      // K_e[h = k][n = col]
                    Rs[kk][c] = v;
                }
            }
        }
        __syncthreads();
#pragma unroll 4
        for (int kk = 0; kk < 16; ++kk) {
            float l[kBU], r[kBU];
#pragma unroll
            for (int u = 0; u < kBU; ++u) {
                l[u] = Ls[kk][ty * kBU + u];
                r[u] = Rs[kk][tx * kBU + u];
            }
#pragma unroll
            for (int u = 0; u < kBU; ++u)
#pragma unroll
                for (int v = 0; v < kBU; ++v) acc[u][v] = fmaf(l[u], r[v], acc[u][v]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < kBU; ++u) {
        const int pr = r0 + ty * kBU + u;
        if (pr >= p1) continue;
        const uint64_t mask = p.pair_mask[pr];
#pragma unroll
        for (int v = 0; v < kBU; ++v) {
            const int col = c0 + tx * kBU + v;
            if (col >= cols) continue;
            const float a = acc[u][v];
            if constexpr (MODE == 0) {
                const bool on = (mask >> (col / p.M)) & 1ull;
                p.act[(size_t)pr * p.H + col] = on ? gelu_erf(a) : 0.f;
                p.da[(size_t)pr * p.H + col] = on ? gelu_grad_erf(a) : 0.f;
            } else if constexpr (MODE == 2) {
                float* g = p.da + (size_t)pr * p.H + col;
                *g = a * *g;
            } else {
                p.dxp[(size_t)pr * p.d + col] = a;
            }
        }
    }
}

// Per token: the router-logit gradients dz (dz0 for W_shr through alpha,
// dl_j for W_j through the softmax) and dX = the sum of the token's dx_pair
// plus sum_j dz_j W_j. A workgroup takes kTokTile tokens: their dz first
// (one thread per (token, slot)), kept in LDS and written out for the
// router's weight gradient; then each thread takes columns n, holds W_j[n]
// for 16 j at a time in registers and adds their terms to all the tile's
// tokens. Fixed summation order: the pairs in slot order, then j = 0..K.
constexpr int kTokTile = 16;
constexpr int kDzRow = 80;   // K+1 <= 65, rounded up to whole groups of 16

__global__ __launch_bounds__(256) void bwd_token_kernel(BwdParams p) {
    __shared__ float dzs[kTokTile][kDzRow];
    __shared__ float sdp_s[kTokTile];
    __shared__ int pofs[kTokTile][kDzRow];   // the tile's pairs by slot (0 past a token's k)
    const int K1 = p.K + 1;
    const int t0 = blockIdx.x * kTokTile;
    const int nt = min(kTokTile, p.N - t0);
    for (int x = threadIdx.x; x < kTokTile * kDzRow; x += blockDim.x) dzs[x / kDzRow][x % kDzRow] = 0.f;
    // sum_m p_m dp_m with dp nonzero for the k selected experts
    if ((int)threadIdx.x < nt) {
        const int t = t0 + threadIdx.x;
        const int k = p.nres[t];
        const int* of = p.pair_of + (size_t)t * K1;
        float sdp = 0.f;
        for (int i = 0; i < k; ++i) sdp = fmaf(p.wts[(size_t)t * p.K + i], p.dcoef[of[1 + i]], sdp);
        sdp_s[threadIdx.x] = sdp;
    }
    __syncthreads();
    // Slot 0: alpha = tau + (1 - 2 tau) sigma(z0), so dz0 = dcoef_shr (1 - 2
    // tau) sigma (1 - sigma), sigma recovered from alpha. Slot i + 1: p_i =
    // s_{q_i}, dl_{q_i} = p_i (dp_{q_i} - sum_m p_m dp_{q_m}). Padded tokens
    // get zeros (slot i then stands for j = i).
    for (int x = threadIdx.x; x < nt * K1; x += blockDim.x) {
        const int tt = x / K1, i = x - tt * K1, t = t0 + tt;
        const int k = p.nres[t];
        float v = 0.f;
        int j = i;
        if (k > 0) {
            const int* of = p.pair_of + (size_t)t * K1;
            if (i == 0) {
                if (p.alpha_adaptive) {
                    const float sg = (p.alpha[t] - p.tau) / p.one_minus_2tau;
                    v = p.dcoef[of[0]] * p.one_minus_2tau * sg * (1.f - sg);
                }
            } else {
                const float pi = p.wts[(size_t)t * p.K + i - 1];
                const float dpi = (i - 1 < k) ? p.dcoef[of[i]] : 0.f;
                v = pi * (dpi - sdp_s[tt]);
                j = p.eids[(size_t)t * p.K + i - 1];
            }
        }
        dzs[tt][j] = v;
        p.dz[(size_t)t * K1 + j] = v;
    }
    __syncthreads();
    // dX, 4 columns per thread: the pair rows slot by slot across the tile's
    // tokens, then the router terms 8 j at a time with W_j[n..n+3] in
    // registers. The tile's pair indices are staged in LDS and a slot's 16
    // row loads are issued unconditionally (slots a token lacks re-read pair
    // 0 and add nothing), so they are all in flight together.
    int kk[kTokTile];
    int kmax = 0;
#pragma unroll
    for (int tt = 0; tt < kTokTile; ++tt) {
        kk[tt] = tt < nt ? p.nres[t0 + tt] : 0;
        kmax = max(kmax, kk[tt]);
    }
    for (int x = threadIdx.x; x < kTokTile * K1; x += blockDim.x) {
        const int tt = x / K1, i = x - tt * K1;
        const int k = tt < nt ? p.nres[t0 + tt] : 0;
        pofs[tt][i] = (k > 0 && i <= k) ? p.pair_of[(size_t)(t0 + tt) * K1 + i] : 0;
    }
    __syncthreads();
    const int nslot = (kmax > 0) ? kmax + 1 : 0;   // kmax = 0: every token of the tile is padded
    for (int n = 4 * (int)threadIdx.x; n < p.d; n += 4 * (int)blockDim.x) {
        f32x4 acc[kTokTile];
#pragma unroll
        for (int tt = 0; tt < kTokTile; ++tt) acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int i = 0; i < nslot; ++i) {
            f32x4 v[kTokTile];
#pragma unroll
            for (int tt = 0; tt < kTokTile; ++tt)
                v[tt] = *reinterpret_cast<const f32x4*>(p.dxp + (size_t)pofs[tt][i] * p.d + n);
#pragma unroll
            for (int tt = 0; tt < kTokTile; ++tt)
                if (i <= kk[tt] && kk[tt] > 0) acc[tt] += v[tt];
        }
        for (int j0 = 0; j0 < K1; j0 += 8) {
            f32x4 w[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                w[u] = (j0 + u < K1) ? *reinterpret_cast<const f32x4*>(p.Wr + (size_t)(j0 + u) * p.d + n)
                                     : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int tt = 0; tt < kTokTile; ++tt)
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const float z = dzs[tt][j0 + u];
#pragma unroll
                    for (int q = 0; q < 4; ++q) acc[tt][q] = fmaf(z, w[u][q], acc[tt][q]);
                }
        }
#pragma unroll
        for (int tt = 0; tt < kTokTile; ++tt)
            if (tt < nt)
                *reinterpret_cast<f32x4*>(p.dX + (size_t)(t0 + tt) * p.d + n) =
                    kk[tt] > 0 ? acc[tt] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
}

// dW_router[j][n] = sum_t dz[t][j] x_t[n] in two passes: partial sums over
// kRouterChunks slices of the tokens (blockIdx.z), then their sum in slice
// order. One wave per (128 columns, 32 j, slice), on the matrix cores in
// fp32 (v_mfma_f32_32x32x2_f32, two tokens per step, four products side by
// side): lane l brings dz[t + l / 32][j0 + l % 32] as its A value and
// x_{t + l / 32}[n0 + 4 (l % 32) + b] as its B value of product b, so column
// cc of product b stands for n = n0 + 4 cc + b and one load gives a lane its
// four B values. The loads of the next 16 tokens are in flight while the
// current 16 are multiplied.
constexpr int kRouterChunks = 256;
constexpr int kRouterCols = 128;

// Four consecutive values of a layer-format tensor: the raw bytes (8 for
// bf16, 16 for fp32), then as floats.
template <bool BF16>
using raw4_t = typename std::conditional<BF16, uint2, f32x4>::type;

template <bool BF16>
__device__ __forceinline__ raw4_t<BF16> ld_raw4(const void* p, size_t i) {
    if constexpr (BF16) return *reinterpret_cast<const uint2*>(static_cast<const u16*>(p) + i);
    else return *reinterpret_cast<const f32x4*>(static_cast<const float*>(p) + i);
}

template <bool BF16>
__device__ __forceinline__ f32x4 raw4_f32(raw4_t<BF16> r) {
    if constexpr (BF16)
        return f32x4{__uint_as_float(r.x << 16), __uint_as_float(r.x & 0xffff0000u), __uint_as_float(r.y << 16),
                     __uint_as_float(r.y & 0xffff0000u)};
    else return r;
}

template <bool BF16>
__global__ __launch_bounds__(64) void bwd_router_kernel(BwdParams p) {
    constexpr int U = 8;   // steps (two tokens each) per batch of loads
    const int K1 = p.K + 1;
    const int lane = (int)threadIdx.x, lr = lane & 31, lh = lane >> 5;
    const int n0 = (int)blockIdx.x * kRouterCols, j0 = (int)blockIdx.y * 32, c = (int)blockIdx.z;
    const int t0 = (int)((int64_t)c * p.N / kRouterChunks), t1 = (int)((int64_t)(c + 1) * p.N / kRouterChunks);
    const int j = j0 + lr, n = n0 + 4 * lr;
    const bool jok = j < K1, nok = n < p.d;   // d % 4 == 0: a lane's 4 columns are all in or all out
    // Loads are issued for every lane and step (out-of-range ones read a
    // valid element of the slice, row t1 - 1, and are zeroed afterwards), so
    // a batch's loads are all in flight together.
    const int jc = jok ? j : 0, nc = nok ? n : 0;
    f32x16 acc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = f32x16{};
    float a[2][U];
    raw4_t<BF16> x[2][U];
    auto load = [&](int t, int set) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int tt = min(t + 2 * u + lh, t1 - 1);
            a[set][u] = p.dz[(size_t)tt * K1 + jc];
            x[set][u] = ld_raw4<BF16>(p.X, (size_t)tt * p.d + nc);
        }
    };
    auto multiply = [&](int t, int set) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool ok = t + 2 * u + lh < t1;
            const float av = (ok && jok) ? a[set][u] : 0.f;
            const f32x4 xv = raw4_f32<BF16>(x[set][u]);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                acc[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, nok ? xv[q] : 0.f, acc[q], 0, 0, 0);
        }
    };
    if (t0 < t1) load(t0, 0);
    for (int t = t0; t < t1; t += 4 * U) {
        if (t + 2 * U < t1) load(t + 2 * U, 1);
        multiply(t, 0);
        if (t + 2 * U >= t1) break;
        if (t + 4 * U < t1) load(t + 4 * U, 0);
        multiply(t + 2 * U, 1);
    }
    // Lane l holds rows (v / 4) 8 + 4 (l / 32) + v % 4 of column l % 32 of
    // each product.
    if (nok)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int r = j0 + (v >> 2) * 8 + lh * 4 + (v & 3);
            if (r < K1)
                *reinterpret_cast<f32x4*>(p.rpart + ((size_t)c * K1 + r) * p.d + n) =
                    f32x4{acc[0][v], acc[1][v], acc[2][v], acc[3][v]};
        }
}

__global__ __launch_bounds__(256) void bwd_router_sum_kernel(BwdParams p) {
    const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t n = (size_t)(p.K + 1) * p.d;
    if (item >= n) return;
    float s = 0.f;
    for (int c = 0; c < kRouterChunks; ++c) s += p.rpart[(size_t)c * n + item];
    p.dWr[item] = s;
}

// Weight gradients of expert e as two fp32 GEMMs over its pairs:
//   dW_up[e][h][n]   = sum_pr da[pr][h] x_{tok(pr)}[n]
//   dW_down[e][n][h] = sum_pr w_pr dy_{tok(pr)}[n] act[pr][h]
// blockIdx.z = e, blockIdx.y picks the product (0: up, 1: down); one
// kBT x kBT output tile per workgroup (rows: h for up, n for down). The sum
// runs over the tokens in order, 16 per LDS step, each step taking the
// step's pairs with expert e (a token has at most one), so it is the same on
// every call (the segment order of the pairs follows the routing kernel's
// atomics).
__global__ __launch_bounds__(256) void bwd_wgrad_kernel(BwdParams p, int tiles_h, int tiles_d) {
    __shared__ float Ls[16][kBT + 1];   // pair x output-row operand
    __shared__ float Rs[16][kBT + 1];   // pair x output-column operand
    __shared__ int prs[16];             // the step's pairs with expert e (-1: none)
    const int e = blockIdx.z, up = blockIdx.y == 0;
    const int rows = up ? p.H : p.d, cols = up ? p.d : p.H;
    const int tr = up ? tiles_h : tiles_d, tc = up ? tiles_d : tiles_h;
    const int tile = blockIdx.x;
    if (tile >= tr * tc) return;
    const int r0 = (tile / tc) * kBT, c0 = (tile % tc) * kBT;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    // Channel blocks of this tile (rows h for up, columns h for down): a
    // 16-token step whose pairs run none of them adds exact zeros and is
    // skipped.
    const uint64_t tmask = up ? channel_blocks(r0, min(r0 + kBT, rows), p.M)
                              : channel_blocks(c0, min(c0 + kBT, cols), p.M);
    float acc[kBU][kBU] = {};
    for (int q0 = 0; q0 < p.N; q0 += 16) {
        if (threadIdx.x < 16) {
            const int t = q0 + threadIdx.x;
            int pr = -1;
            const int k = t < p.N ? p.nres[t] : 0;
            if (k > 0) {
                if (e == 0) {
                    pr = p.pair_of[(size_t)t * (p.K + 1)];
                } else {
                    for (int i = 0; i < k; ++i)
                        if (p.eids[(size_t)t * p.K + i] == e) {
                            pr = p.pair_of[(size_t)t * (p.K + 1) + 1 + i];
                            break;
                        }
                }
            }
            prs[threadIdx.x] = pr;
        }
        __syncthreads();
        uint64_t cu = 0;
        for (int j = 0; j < 16; ++j)
            if (prs[j] >= 0) cu |= p.pair_mask[prs[j]];
        if ((cu & tmask) == 0) {
            __syncthreads();   // every thread has read prs before it is rewritten
            continue;
        }
        for (int i = threadIdx.x; i < 16 * kBT; i += blockDim.x) {
            const int pi = i / kBT, x = i % kBT, pr = prs[pi];
            float lv = 0.f, rv = 0.f;
            if (pr >= 0) {
                const int t = q0 + pi;
                if (up) {
                    if (r0 + x < rows) lv = p.da[(size_t)pr * p.H + r0 + x];
                    if (c0 + x < cols) rv = ld_f32(p.X, (size_t)t * p.d + c0 + x);
                } else {
                    if (r0 + x < rows) lv = p.pw[pr] * ld_f32(p.dY, (size_t)t * p.d + r0 + x);
                    if (c0 + x < cols) rv = p.act[(size_t)pr * p.H + c0 + x];
                }
            }
            Ls[pi][x] = lv;
            Rs[pi][x] = rv;
        }
        __syncthreads();
#pragma unroll 4
        for (int pi = 0; pi < 16; ++pi) {
            float l[kBU], r[kBU];
#pragma unroll
            for (int u = 0; u < kBU; ++u) {
                l[u] = Ls[pi][ty * kBU + u];
                r[u] = Rs[pi][tx * kBU + u];
            }
#pragma unroll
            for (int u = 0; u < kBU; ++u)
#pragma unroll
                for (int v = 0; v < kBU; ++v) acc[u][v] = fmaf(l[u], r[v], acc[u][v]);
        }
        __syncthreads();
    }
    float* out = up ? p.dWup + (size_t)e * p.H * p.d : p.dWdown + (size_t)e * p.d * p.H;
#pragma unroll
    for (int u = 0; u < kBU; ++u) {
        const int r = r0 + ty * kBU + u;
        if (r >= rows) continue;
#pragma unroll
        for (int v = 0; v < kBU; ++v) {
            const int c = c0 + tx * kBU + v;
            if (c < cols) out[(size_t)r * cols + c] = acc[u][v];
        }
    }
}

// Gram diversity loss of the augmented router (Eq. diversity-loss):
// L_div = || W W^T - I ||_F over the K+1 router rows W (W_shr, W_1..W_K),
// and dW += lambda (2 / L_div) (W W^T - I) W (none when L_div = 0). fp64
// throughout (the products of fp32 values are exact), every sum in a fixed
// order, so the result is the same on every call.
struct DivParams {
    int K1, d;
    const float* W;      // [K+1, d]
    double* G;           // [K+1, K+1] workspace
    double* Ls;          // [1] workspace: L_div
    float* loss;         // [1]
    float* dW;           // [K+1, d], updated
    float lambda;
};

// G[i][j] = W_i . W_j, one wave per pair i <= j (lanes take n = lane + 64 t,
// then a fixed shuffle tree).
__global__ __launch_bounds__(256) void div_gram_kernel(DivParams p) {
    const int w = blockIdx.x * 4 + (int)(threadIdx.x >> 6);
    const int npair = p.K1 * (p.K1 + 1) / 2;
    if (w >= npair) return;
    int i = 0, rem = w;
    while (rem >= p.K1 - i) {
        rem -= p.K1 - i;
        ++i;
    }
    const int j = i + rem;
    const float* a = p.W + (size_t)i * p.d;
    const float* b = p.W + (size_t)j * p.d;
    double s = 0.0;
    for (int n = lane_id(); n < p.d; n += kWave) s = fma((double)a[n], (double)b[n], s);
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane_id() == 0) {
        p.G[(size_t)i * p.K1 + j] = s;
        p.G[(size_t)j * p.K1 + i] = s;
    }
}

// L_div from G (one workgroup of 256: strided partial sums, then a fixed
// tree in LDS).
__global__ __launch_bounds__(256) void div_loss_kernel(DivParams p) {
    __shared__ double part[256];
    const int n = p.K1 * p.K1;
    double s = 0.0;
    for (int x = threadIdx.x; x < n; x += 256) {
        const double v = p.G[x] - ((x / p.K1 == x % p.K1) ? 1.0 : 0.0);
        s = fma(v, v, s);
    }
    part[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) part[threadIdx.x] += part[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double L = sqrt(part[0]);
        *p.Ls = L;
        *p.loss = (float)L;
    }
}

// dW[i][n] += lambda (2 / L) sum_j (G - I)[i][j] W[j][n], one thread per (i, n).
__global__ __launch_bounds__(256) void div_grad_kernel(DivParams p) {
    const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (item >= (size_t)p.K1 * p.d) return;
    const double L = *p.Ls;
    if (L == 0.0 || p.lambda == 0.0f) return;
    const int i = (int)(item / p.d), n = (int)(item - (size_t)i * p.d);
    double g = 0.0;
    for (int j = 0; j < p.K1; ++j)
        g = fma(p.G[(size_t)i * p.K1 + j] - (i == j ? 1.0 : 0.0), (double)p.W[(size_t)j * p.d + n], g);
    p.dW[item] = (float)((double)p.dW[item] + (double)p.lambda * (2.0 / L) * g);
}

}  // namespace unifmoe
