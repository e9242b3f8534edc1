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
// Copies of the per-expert pair totals that the routing tiles add into
// (spreading same-address atomics); the permutation sums them.
constexpr int kExpCopies = 16;
// Copies of each (expert, mask key) bin of the pair sort: token tile q counts
// its pairs and takes their slots in copy q % kBinCopies, so that no counter
// sees more than a share of its bin's atomics (atomics on one cache line
// serialize at the L2); a bin's slots are its copies' ranges in copy order.
constexpr int kBinCopies = 8;
// XCDs of an MI355X (each with its own L2); the persistent GEMMs keep one
// tile queue per XCD.
constexpr int kXcds = 8;

// The counter of copy c of bin `bin` among nbin bins: the copies of a bin lie
// nbin counters apart, on different cache lines (and L2 channels), so a bin
// that many pairs share spreads its atomics over kBinCopies lines.
__host__ __device__ __forceinline__ size_t bin_counter(int bin, int c, int nbin) {
    return (size_t)c * (size_t)nbin + (size_t)bin;
}

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

// D = A(32x16) * B(16x32) + C on the matrix cores. Lane l supplies row
// (A) / column (B) l % 32 and the 8 consecutive k of group l / 32; element
// 4 j + i of the accumulator holds D[8 j + 4 (l / 32) + i][l % 32].
typedef float f32x16 __attribute__((ext_vector_type(16)));
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// The same product with fp16 operands (v_mfma_f32_32x32x16_f16; lane layout
// as above).
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ f16x8 as_f16x8(u32x4 v) { return __builtin_bit_cast(f16x8, v); }
__device__ __forceinline__ f32x16 mfma32x32x16_f16(f16x8 a, f16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// GELU(a) = a/2 (1 + erf(a / sqrt 2)), exact erf form (library erff).
__device__ __forceinline__ float gelu_erf(float a) {
    return 0.5f * a * (1.0f + erff(a * 0.7071067811865475244f));
}

// GELU(a) = a Phi(a) = a / 2 + |a| (1/2 - Phi(-|a|)), with Phi(-y) = 2^Q(y) and
// Q(y) = log2 Phi(-y) replaced by a degree-7 polynomial fitted on [0, 6]
// (gelu_coeffs.py prints kGeluQ), evaluated at |a|: one exp2 and ten other
// vector instructions. Past the fit range the polynomial keeps falling
// (Q(6) = -29.9, its leading coefficient is negative, and in fp32 it reaches
// -inf for huge |a|), so 2^Q stays below 2^-29.9 there, as Phi(-|a|) does.
// In fp32 the error is below 1e-5 |GELU(a)| + 3e-8 |a| for |a| < 6 (the
// second term, from rounding 1/2 - Phi(-|a|), matters only in the far
// negative tail) and below 5e-7 everywhere (|a| 2^-29.9 bounds it past 6);
// used where the result is rounded to fp16 (relative spacing 2^-11), far
// above that.
constexpr float kGeluQ[8] = {-9.999869466e-01f, -1.151324511e+00f, -4.582976401e-01f, -5.411815643e-02f,
                             8.582305163e-03f,  -9.488553624e-04f, 6.385870802e-05f,  -1.944835731e-06f};
constexpr float kGeluQMax = 6.0f;
__device__ __forceinline__ float gelu_exp2poly(float a) {
    // |a| is a source modifier of the first fma; a NaN input yields NaN.
    const float y = fabsf(a);
    float q = fmaf(kGeluQ[7], y, kGeluQ[6]);
    q = fmaf(q, y, kGeluQ[5]);
    q = fmaf(q, y, kGeluQ[4]);
    q = fmaf(q, y, kGeluQ[3]);
    q = fmaf(q, y, kGeluQ[2]);
    q = fmaf(q, y, kGeluQ[1]);
    q = fmaf(q, y, kGeluQ[0]);
    // a Phi(a) = a / 2 + |a| (1/2 - Phi(-|a|)), which keeps GELU(+inf) = +inf.
    return fmaf(fabsf(a), 0.5f - __builtin_amdgcn_exp2f(q), 0.5f * a);
}

// GELU(a) as gelu_exp2poly and its derivative Phi(a) + a phi(a) from the
// same fitted Phi(-|a|) = 2^Q(|a|): Phi(a) = 1 - Phi(-a) for a >= 0, and
// phi(a) = 2^(-a^2 log2(e) / 2) / sqrt(2 pi). In fp32 the derivative is
// within 5e-6 of the exact one (the fit's error at 0, where Phi(-0) = 1/2
// comes out 4.5e-6 high), far below the fp16 rounding it then gets.
__device__ __forceinline__ void gelu_exp2poly_grad(float a, float& g, float& gp) {
    const float y = __builtin_amdgcn_fmed3f(fabsf(a), 0.0f, kGeluQMax);
    float q = fmaf(kGeluQ[7], y, kGeluQ[6]);
    q = fmaf(q, y, kGeluQ[5]);
    q = fmaf(q, y, kGeluQ[4]);
    q = fmaf(q, y, kGeluQ[3]);
    q = fmaf(q, y, kGeluQ[2]);
    q = fmaf(q, y, kGeluQ[1]);
    q = fmaf(q, y, kGeluQ[0]);
    const float P = __builtin_amdgcn_exp2f(q);
    g = fmaf(fabsf(a), 0.5f - P, 0.5f * a);
    const float phi2 = __builtin_amdgcn_exp2f((-0.7213475204444817f * a) * a);
    gp = fmaf(a * 0.3989422804014327f, phi2, a >= 0.0f ? 1.0f - P : P);
}

// Two fp32 -> packed bf16 pair (round to nearest even, one gfx950
// v_cvt_pk_bf16_f32); `lo` lands in the low half.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    bf16x2 v;
    v[0] = (__bf16)lo;
    v[1] = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

// Two fp32 -> packed fp16 pair, each rounded to nearest even (values beyond
// the fp16 range become infinities); `lo` lands in the low half.
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    f16x2 v;
    v[0] = (_Float16)lo;
    v[1] = (_Float16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

// A packed fp16 pair (pack_f16x2's layout) as two fp32 values (exact).
__device__ __forceinline__ void unpack_f16x2(uint32_t v, float& lo, float& hi) {
    const f16x2 h = __builtin_bit_cast(f16x2, v);
    lo = (float)h[0];
    hi = (float)h[1];
}

// Column j of an 8 x 8 block of 16-bit values held as eight rows of 16
// bytes (v[q] = row q): the eight values of rows 0..7 at position j, as one
// 16-byte row (row q in half q % 2 of word q / 2).
__device__ __forceinline__ u32x4 column8(const u32x4 (&v)[8], int j) {
    u32x4 o;
    const int w = j >> 1;
#pragma unroll
    for (int m = 0; m < 4; ++m)
        o[m] = (j & 1) ? ((v[2 * m][w] >> 16) | (v[2 * m + 1][w] & 0xffff0000u))
                       : ((v[2 * m][w] & 0xffffu) | (v[2 * m + 1][w] << 16));
    return o;
}

// d GELU / da = Phi(a) + a phi(a) (library erff and expf).
__device__ __forceinline__ float gelu_grad_erf(float a) {
    return 0.5f * (1.0f + erff(a * 0.7071067811865475244f)) + a * 0.3989422804014327f * expf(-0.5f * a * a);
}

// Load of a wave-uniform address through the constant address space, so it
// becomes a scalar-cache load (lgkmcnt) instead of a vector load whose wait
// would also drain in-flight vector-memory copies. Only for data that no
// store of the running kernel touches.
__device__ __forceinline__ int ld_uniform(const int* p) {
    return *(const __attribute__((address_space(4))) int*)p;
}

__device__ __forceinline__ uint64_t ld_uniform64(const uint64_t* p) {
    return *(const __attribute__((address_space(4))) uint64_t*)p;
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int mask) {
    const uint32_t lo = __shfl_xor((uint32_t)v, mask), hi = __shfl_xor((uint32_t)(v >> 32), mask);
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }
__device__ __forceinline__ uint64_t lanes_below() {
    return (lane_id() == 0) ? 0ull : (~0ull >> (kWave - lane_id()));
}

__host__ __device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Sort key of a B-bit block mask: its top kb bits (kb <= 16), replaced by
// their rank in the reflected Gray code sequence, so that key order puts
// masks that differ in one block next to each other.
__device__ __forceinline__ int mask_key(uint64_t mask, int B, int kb) {
    uint32_t v = (uint32_t)(B > kb ? (mask >> (B - kb)) : mask);
    v ^= v >> 1;
    v ^= v >> 2;
    v ^= v >> 4;
    v ^= v >> 8;
    return (int)v;
}

// put(i, get(i)) for i in [0, n), the workgroup's threads striding over i;
// each thread issues a batch of 8 gets (global loads) before any put, so the
// loads' latencies overlap instead of adding up one per iteration.
template <class Get, class Put>
__device__ __forceinline__ void batched_copy(int n, Get get, Put put) {
    const int T = blockDim.x;
    for (int i0 = threadIdx.x; i0 < n; i0 += 8 * T) {
        decltype(get(0)) v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (i0 + u * T < n) v[u] = get(i0 + u * T);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (i0 + u * T < n) put(i0 + u * T, v[u]);
    }
}

// Largest i in [0, n) with off[i] <= x (off ascending, off[0] = 0 <= x).
__device__ __forceinline__ int upper_index(const int* off, int n, int x) {
    int lo = 0, hi = n;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (off[mid] <= x) lo = mid;
        else hi = mid;
    }
    return lo;
}

// Asynchronous copies global -> LDS (gfx950 global_load_lds_dword[x4]): lane
// l of the wave writes its 4 or 16 bytes at lds_base + 4 l or + 16 l, where
// lds_base (in M0) is the same for the whole wave. Completion is tracked by
// vmcnt only. (Measured on gfx950 interleaved with MFMAs, this form sustains
// more copy bandwidth at less MFMA cost than the buffer-load form of the same
// copy.)
// They are issued as inline assembly, so the compiler does not model them:
// a compiler-visible LDS copy makes it wait for every LDS read in flight
// (lgkmcnt(0)) wherever a fragment read is consumed, which defeats reading
// the next k step's fragments ahead. Every consumer of the copied data
// therefore waits explicitly (wait_vmcnt, then a barrier); the compiler's
// own vmcnt waits for its loads can only over-count the copies. M0 is set
// by each copy and used by nothing else in these kernels.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}
// (M0 is a reserved register: clang warns that clobbering it is not
// tracked; the kernels keep no value in M0 across a copy.)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* gsrc, void* lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gsrc), "s"(lds_offset(lds_base))
                 : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* gsrc, void* lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
                 :
                 : "v"(gsrc), "s"(lds_offset(lds_base))
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// Wait until at most N vector-memory operations of this wave are pending.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier for LDS data only: this wave's LDS operations complete,
// then s_barrier. The "memory" clobber keeps the compiler from moving memory
// accesses across it; unlike __syncthreads it does not wait for global
// loads in flight.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until all LDS operations of this wave have completed.
__device__ __forceinline__ void wait_lgkmcnt0() {
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));
}

}  // namespace unifmoe
