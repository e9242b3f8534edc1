// Weighted merge of Eq. output: y = alpha E_shr^S + sum_{i <= k} p_i E_{q_i}^R.
// Each token reads its k + 1 per-expert rows (pair_of) and sums them in a
// fixed order (shared expert first, then q_1..q_k) in fp32, so the result
// does not depend on how pairs were scheduled. Padded rows get zeros.
#pragma once
#include "common.hpp"

namespace unifmoe {

struct CombineParams {
    int N, d, K;
    const void* part;
    const int* pair_of;
    const float* alpha;
    const int* nres;
    const float* wts;
    void* Y;
};

// bf16 output: one thread per 8 consecutive outputs; fp32 per-expert rows
// (two 16-byte loads each), one 16-byte store.
__global__ void combine_bf16_kernel(CombineParams c) {
    const int chunks = c.d >> 3;
    const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (item >= (size_t)c.N * chunks) return;
    const int t = (int)(item / chunks), ch = (int)(item - (size_t)t * chunks);
    const int k = c.nres[t];
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const float* part = static_cast<const float*>(c.part);
    for (int i = 0; i <= k && k > 0; ++i) {
        const float w = (i == 0) ? c.alpha[t] : c.wts[(size_t)t * c.K + i - 1];
        const int pr = c.pair_of[(size_t)t * (c.K + 1) + i];
        const float* src = part + (size_t)pr * c.d + ch * 8;
        const u32x4 v0 = ld16(src), v1 = ld16(src + 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            acc[q] = fmaf(w, __uint_as_float(v0[q]), acc[q]);
            acc[4 + q] = fmaf(w, __uint_as_float(v1[q]), acc[4 + q]);
        }
    }
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = (uint32_t)f2bf(acc[2 * q]) | ((uint32_t)f2bf(acc[2 * q + 1]) << 16);
    st16(static_cast<u16*>(c.Y) + (size_t)t * c.d + ch * 8, o);
}

// fp32: one thread per output element.
__global__ void combine_f32_kernel(CombineParams c) {
    const size_t item = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (item >= (size_t)c.N * c.d) return;
    const int t = (int)(item / c.d), j = (int)(item - (size_t)t * c.d);
    const int k = c.nres[t];
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
