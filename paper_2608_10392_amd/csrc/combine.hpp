// Weighted merge of Eq. output: y = alpha E_shr^S + sum_{i <= k} p_i E_{q_i}^R.
// Each token reads its k + 1 per-expert rows (pair_of) and sums them in a
// fixed order (shared expert first, then q_1..q_k) in fp32, so the result
// does not depend on how pairs were scheduled. Padded rows get zeros.
#pragma once
#include "common.hpp"

namespace unifmoe {

struct CombineParams {
    int N, d, K;
    int nsplit;            // row buffers per pair (the down-projection's parts), summed in order
    size_t split_stride;   // floats between them
    const void* part;
    const int* pair_of;
    const float* alpha;
    const int* nres;
    const float* wts;
    void* Y;
    const int* totals;     // totals[5] != 0: the routing overflowed the pair capacity (Y = 0)
};

constexpr int kCombineBatch = 6;

// bf16 layers: one thread per 4 consecutive outputs; fp32 per-expert rows
// (one 16-byte load each, per part with SPLIT), one 8-byte bf16 store. (Four
// outputs per thread keep more rows in flight per CU than eight: 10% less
// time on the 50k-token d = 768 layer.)
template <bool SPLIT>
__global__ void combine_bf16_kernel(CombineParams c) {
    const int chunks = c.d >> 2;
    const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (item >= (size_t)c.N * chunks) return;
    const int t = (int)(item / chunks), ch = (int)(item - (size_t)t * chunks);
    // past the pair capacity no expert row exists: Y = 0
    const int k = ld_uniform(c.totals + 5) ? 0 : c.nres[t];
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    const float* part = static_cast<const float*>(c.part);
    const int* of = c.pair_of + (size_t)t * (c.K + 1);
    const float* wt = c.wts + (size_t)t * c.K;
    // Rows in batches of kCombineBatch: the weights and pair indices of a
    // batch, then its rows, are loaded before any is used (the latencies
    // overlap); the sum still runs in the fixed order. The first batch's
    // weights and indices do not wait for k: entries up to K are always
    // readable, and those past k are not used.
    for (int i0 = 0; i0 == 0 || (i0 <= k && k > 0); i0 += kCombineBatch) {
        float w[kCombineBatch];
        int pr[kCombineBatch];
#pragma unroll
        for (int u = 0; u < kCombineBatch; ++u) {
            const int i = i0 + u;
            const bool in = (i0 == 0) ? i <= c.K : i <= k;
            w[u] = in ? (i == 0 ? c.alpha[t] : wt[i - 1]) : 0.f;
            pr[u] = in ? of[i] : 0;
        }
        if (k == 0) break;
        // The rows are read once and Y written once: non-temporal accesses
        // keep them from displacing cached data.
        f32x4 v[kCombineBatch];
#pragma unroll
        for (int u = 0; u < kCombineBatch; ++u)
            v[u] = (i0 + u <= k)
                       ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(part + (size_t)pr[u] * c.d + ch * 4))
                       : f32x4{0.f, 0.f, 0.f, 0.f};
        for (int sp = 1; SPLIT && sp < c.nsplit; ++sp) {
#pragma unroll
            for (int u = 0; u < kCombineBatch; ++u)
                if (i0 + u <= k)
                    v[u] += __builtin_nontemporal_load(
                        reinterpret_cast<const f32x4*>(part + sp * c.split_stride + (size_t)pr[u] * c.d + ch * 4));
        }
#pragma unroll
        for (int u = 0; u < kCombineBatch; ++u) {
            if (i0 + u <= k) {
#pragma unroll
                for (int q = 0; q < 4; ++q) acc[q] = fmaf(w[u], v[u][q], acc[q]);
            }
        }
    }
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    u32x2 o;
    o[0] = (uint32_t)f2bf(acc[0]) | ((uint32_t)f2bf(acc[1]) << 16);
    o[1] = (uint32_t)f2bf(acc[2]) | ((uint32_t)f2bf(acc[3]) << 16);
    __builtin_nontemporal_store(o, reinterpret_cast<u32x2*>(static_cast<u16*>(c.Y) + (size_t)t * c.d + ch * 4));
}

// fp32: one thread per output element.
__global__ void combine_f32_kernel(CombineParams c) {
    const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (item >= (size_t)c.N * c.d) return;
    const int t = (int)(item / c.d), j = (int)(item - (size_t)t * c.d);
    const int k = ld_uniform(c.totals + 5) ? 0 : c.nres[t];   // past the pair capacity: Y = 0
    const float* part = static_cast<const float*>(c.part);
    float acc = 0.f;
    for (int i = 0; i <= k && k > 0; ++i) {
        const float w = (i == 0) ? c.alpha[t] : c.wts[(size_t)t * c.K + i - 1];
        const int pr = c.pair_of[(size_t)t * (c.K + 1) + i];
        acc = fmaf(w, part[(size_t)pr * c.d + j], acc);
    }
    static_cast<float*>(c.Y)[item] = acc;
}

}  // namespace unifmoe
