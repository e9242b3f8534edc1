// Counts of Eq. block-compute over a routing record: histograms of b and k,
// tokens per expert, sums of b, k and C_B = b + k (B - b). Per-workgroup LDS
// histograms, then one 64-bit atomic per bin and workgroup.
#pragma once
#include "common.hpp"

namespace unifmoe {

// Layout of the device counters (unsigned 64-bit words).
constexpr int kStN = 0, kStHistB = 1, kStHistK = 66, kStExp = 131, kStSumB = 196, kStSumK = 197,
              kStSumCB = 198, kStWords = 199;

struct StatsParams {
    int N, K, B;
    const uint8_t* valid;
    const int* nsh;
    const int* nres;
    const int* eids;
    unsigned long long* out;
};

__global__ __launch_bounds__(256) void stats_kernel(StatsParams s) {
    __shared__ unsigned int hb[65], hk[65], he[65];
    __shared__ unsigned long long sums[4];
    for (int i = threadIdx.x; i < 65; i += blockDim.x) hb[i] = hk[i] = he[i] = 0u;
    if (threadIdx.x < 4) sums[threadIdx.x] = 0ull;
    __syncthreads();
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < s.N; t += gridDim.x * blockDim.x) {
        if (s.valid != nullptr && s.valid[t] == 0) continue;
        const int b = s.nsh[t], k = s.nres[t];
        atomicAdd(&hb[b], 1u);
        atomicAdd(&hk[k], 1u);
        atomicAdd(&he[0], 1u);
        for (int i = 0; i < k; ++i) atomicAdd(&he[s.eids[(size_t)t * s.K + i]], 1u);
        atomicAdd(&sums[0], 1ull);
        atomicAdd(&sums[1], (unsigned long long)b);
        atomicAdd(&sums[2], (unsigned long long)k);
        atomicAdd(&sums[3], (unsigned long long)(b + k * (s.B - b)));
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 65; i += blockDim.x) {
        if (hb[i]) atomicAdd(&s.out[kStHistB + i], (unsigned long long)hb[i]);
        if (hk[i]) atomicAdd(&s.out[kStHistK + i], (unsigned long long)hk[i]);
        if (he[i]) atomicAdd(&s.out[kStExp + i], (unsigned long long)he[i]);
    }
    if (threadIdx.x == 0) {
        atomicAdd(&s.out[kStN], sums[0]);
        atomicAdd(&s.out[kStSumB], sums[1]);
        atomicAdd(&s.out[kStSumK], sums[2]);
        atomicAdd(&s.out[kStSumCB], sums[3]);
    }
}

// Work a bf16 forward executed, from its workspace tables: out[0] the block
// count of every 32-row MFMA group of the down-projection's row tiles, summed
// (each counts 32 rows x M x d x 2 FLOPs). One thread per row tile.
__global__ __launch_bounds__(256) void work_kernel(const uint64_t* __restrict__ rt_masks, const int* __restrict__ totals,
                                                   int groups, unsigned long long* out) {
    const int nrt = totals[4];
    unsigned long long n = 0;
    for (int rt = blockIdx.x * blockDim.x + threadIdx.x; rt < nrt; rt += gridDim.x * blockDim.x)
        for (int g = 0; g < groups; ++g) n += (unsigned long long)__popcll(rt_masks[(size_t)rt * (groups + 1) + g]);
    for (int o = 32; o > 0; o >>= 1) n += __shfl_xor(n, o);
    if ((threadIdx.x & 63) == 0 && n) atomicAdd(out, n);
}

}  // namespace unifmoe
