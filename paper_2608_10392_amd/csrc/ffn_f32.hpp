// fp32 expert path (Eq. block-expert-output, fp32 end to end): one
// workgroup evaluates one pair at a time, first the GELU activations of the
// pair's active channels into LDS, then the down-projection over those
// channels, with sequential fp32 FMA dot products. Sized for small layers
// (H = B M <= 16384 floats of LDS); the bf16 matrix-core path is the
// throughput path.
#pragma once
#include "common.hpp"

namespace unifmoe {

struct PairF32Params {
    int d, M, B, H;
    const float* X;
    const float* Wup;    // [K+1][H][d]
    const float* Wdown;  // [K+1][d][H]
    float* part;         // [pairs][d]
    const int* pair_token;
    const int* pair_expert;
    const uint64_t* pair_mask;
    const int* totals;   // [0] pairs, [5] nonzero: more pairs than the buffers hold (nothing to run)
    const float* b_up;   // [K+1][H] biases added before the GELU, or null
};

__global__ __launch_bounds__(256) void pair_ffn_f32_kernel(PairF32Params p) {
    extern __shared__ float g_act[];
    const int P = p.totals[5] ? 0 : p.totals[0];
    for (int pr = blockIdx.x; pr < P; pr += gridDim.x) {
        const int e = p.pair_expert[pr], t = p.pair_token[pr];
        const uint64_t m = p.pair_mask[pr];
        const float* x = p.X + (size_t)t * p.d;
        const float* Wu = p.Wup + (size_t)e * p.H * p.d;
        __syncthreads();
        for (int h = threadIdx.x; h < p.H; h += blockDim.x) {
            float a = 0.f;
            if ((m >> (h / p.M)) & 1ull) {
                const float* w = Wu + (size_t)h * p.d;
                for (int i = 0; i < p.d; ++i) a = fmaf(x[i], w[i], a);
                if (p.b_up != nullptr) a += p.b_up[(size_t)e * p.H + h];
                a = gelu_erf(a);
            }
            g_act[h] = a;
        }
        __syncthreads();
        const float* Wd = p.Wdown + (size_t)e * p.d * p.H;
        for (int j = threadIdx.x; j < p.d; j += blockDim.x) {
            const float* w = Wd + (size_t)j * p.H;
            float s = 0.f;
            for (int c = 0; c < p.B; ++c) {
                if (!((m >> c) & 1ull)) continue;
                for (int h = c * p.M; h < (c + 1) * p.M; ++h) s = fmaf(g_act[h], w[h], s);
            }
            p.part[(size_t)pr * p.d + j] = s;
        }
    }
}

}  // namespace unifmoe
