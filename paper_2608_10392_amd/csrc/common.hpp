// Shared device helpers for the gfx950 kernels: bf16 conversion, MFMA
// operand types, wave64 ballots.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace unifmoe {

typedef uint16_t u16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(u16 v) { return __uint_as_float(((uint32_t)v) << 16); }

// fp32 -> bf16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ u16 f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u16)((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (u16)(u >> 16);
}

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// D = A(16x32) * B(32x16) + C on the matrix cores. Lane l supplies row
// (A) / column (B) l % 16 and the 8 consecutive k of group l / 16; the
// accumulator holds D[4 (l / 16) + r][l % 16] in element r.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// GELU(a) = a/2 (1 + erf(a / sqrt 2)), exact erf form (library erff).
__device__ __forceinline__ float gelu_erf(float a) {
    return 0.5f * a * (1.0f + erff(a * 0.7071067811865475244f));
}

// GELU through the rational-exponential erf approximation of Abramowitz and
// Stegun, Handbook of Mathematical Functions, formula 7.1.26:
//   erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2),
//   t = 1 / (1 + p x), x >= 0, |error| <= 1.5e-7,
// extended to x < 0 by oddness. Branch-free; used where the result is
// rounded to bf16 (relative spacing 2^-8), far above the formula's error.
__device__ __forceinline__ float gelu_as7126(float a) {
    const float x = fabsf(a) * 0.7071067811865475244f;
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
    float poly = fmaf(1.061405429f, t, -1.453152027f);
    poly = fmaf(poly, t, 1.421413741f);
    poly = fmaf(poly, t, -0.284496736f);
    poly = fmaf(poly, t, 0.254829592f);
    poly *= t;
    const float e = __builtin_amdgcn_exp2f(-x * x * 1.4426950408889634f);
    const float erf_abs = fmaf(-poly, e, 1.0f);
    const float erf_x = __builtin_copysignf(erf_abs, a);
    return 0.5f * a * (1.0f + erf_x);
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }
__device__ __forceinline__ uint64_t lanes_below() {
    return (lane_id() == 0) ? 0ull : (~0ull >> (kWave - lane_id()));
}

__host__ __device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Asynchronous 16-byte copy global -> LDS (gfx950 global_load_lds_dwordx4):
// lane l of the wave writes its 16 bytes at lds_base + 16 l, where lds_base
// is the same for the whole wave. Completion is tracked by vmcnt only.
__device__ __forceinline__ void dma16(const void* gsrc, void* lds_base) {
    __builtin_amdgcn_global_load_lds(gsrc, lds_base, 16, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are pending.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Wait until all LDS operations of this wave have completed.
__device__ __forceinline__ void wait_lgkmcnt0() {
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));
}

}  // namespace unifmoe
