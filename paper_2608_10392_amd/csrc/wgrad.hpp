// Expert weight gradients on the matrix cores (the backward of Eq.
// block-expert-output), per (expert e, block c) slab:
//   dW_up[e][c M + h][n]   = sum over the slab's rows r of G[pair(r), c M + h] X[tok(r), n]
//   dW_down[e][n][c M + h] = sum over the slab's rows r of dY[tok(r), n] Hw[pair(r), c M + h]
// where G = d loss / d(x K^T) and Hw = w GELU(x K^T) are the bf16 rows the
// backward's up-projections leave in the layout of the forward's H. Only
// the (pair, block) rows that the forward ran enter, and each sum runs over
// the slab's rows in list order (token order), so the result is the same on
// every call.
//
// Both operands are gathered rows in which the contraction index r is the
// row, while the MFMA takes 8 consecutive r per lane. Each thread loads an
// 8 x 8 block (8 rows, one 16-byte column chunk each), transposes it in
// registers and writes 8 index rows of 8 r to LDS, where a stage is laid out
// index-major: one 128-byte line of 64 r per index (wg_off's swizzle), so
// the fragment reads are the up kernel's. Two stage slots alternate; while
// stage s is multiplied, the rows of stage s + 2 and the list indices of
// stage s + 3 are in flight.
//
// Output tile TQ x TP per workgroup of 8 waves (WQ x WP), where P is the
// output's contiguous index (n for dW_up, h for dW_down) and Q the other.
// P is the MFMA A operand, stored in LDS in wcol order, so each lane
// accumulates 16 consecutive P of one Q and stores them as 64 bytes.
#pragma once
#include "common.hpp"
#include "ffn_bf16.hpp"

namespace unifmoe {

struct WgradParams {
    int d, M, B, H;
    int ntn;                  // n tiles per slab
    const u16* Psrc;          // dW_up: X [N, d];  dW_down: Hw [pairs, H]
    const u16* Qsrc;          // dW_up: G [pairs, H];  dW_down: dY [N, d]
    const int* slab_rows;     // pair of each slab row
    const int* slab_tok;      // token of each slab row
    const int* slab_off;      // first row of each slab in the lists (a multiple of 64)
    const int* slab_count;    // rows of each slab
    float* out;               // dW_up [K+1, H, d] or dW_down [K+1, d, H]
};

// Position in a 32-row group of LDS at which index i (0..31) is stored so
// that the MFMA hands lane l the outputs 16 (l / 32) + 0..15 (wcol's inverse).
__device__ __forceinline__ int wcol_pos(int i) { return (i & 3) | ((i >> 4) << 2) | (((i >> 2) & 3) << 3); }

__host__ __device__ constexpr int wgrad_lds_bytes(int TQ, int TP) { return 2 * (TQ + TP) * Stage::RB; }

// Byte offset of 16-byte chunk c of stage row r: the chunk is rotated by
// bits 1-3, 2-4 and 4-6 of the row. The fragment reads (rows r..r+15 of one
// chunk per 16 lanes) stay free of bank conflicts as with the up kernel's
// layout, and the stores, whose 16 lanes write rows 8 apart with both
// parities (odd chunks store their block's columns in the order j ^ 1),
// fall on nearly all 16 bank groups.
__device__ __forceinline__ uint32_t wg_off(int r, int c) {
    return (uint32_t)r * Stage::RB + ((c ^ (((r >> 1) ^ (r >> 2) ^ (r >> 4)) & 7)) << 4);
}

template <bool UP, int GQ, int GP, int WQ>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void wgrad_kernel(WgradParams p) {
    using S = Stage;
    constexpr int WP = 8 / WQ;
    constexpr int TQ = WQ * GQ * 32, TP = WP * GP * 32;
    constexpr int NCH = (TP + TQ) / 8;        // 16-byte chunks per row of a stage
    constexpr int NU = 8 * NCH;               // (row octet, chunk) units per stage
    constexpr int STAGE = (TP + TQ) * S::RB;
    static_assert(NU <= 512, "one unit per thread");
    extern __shared__ __attribute__((aligned(16))) char lds_wg[];
    const int tid = threadIdx.x, lane = tid & 63, lr = lane & 31, lh = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wq = wave / WP, wp = wave % WP;
    const int slab = blockIdx.x / p.ntn, tn = blockIdx.x - slab * p.ntn;
    const int e = slab / p.B, c = slab - e * p.B;
    const int cnt = ld_uniform(p.slab_count + slab), so = ld_uniform(p.slab_off + slab);
    const int n0 = tn * (UP ? TP : TQ);

    // This thread's unit: rows 8 ro .. 8 ro + 7 of each stage, 16-byte chunk
    // ch of the stage's index range (P indices first, then Q).
    // Threads past the units (whole waves) load like thread 0 and store
    // nothing.
    const bool active = tid < NU;
    const int ro = active ? tid / NCH : 0, ch = active ? tid - (tid / NCH) * NCH : 0;
    const bool isP = ch < TP / 8;
    const int idx0 = isP ? 8 * ch : 8 * (ch - TP / 8);
    const bool tokrows = (UP == isP);            // X and dY rows are tokens; G and Hw rows pairs
    const int* list = (tokrows ? p.slab_tok : p.slab_rows) + so + 8 * ro;
    const u16* src = (isP ? p.Psrc : p.Qsrc) + (tokrows ? n0 : c * p.M) + idx0;
    const size_t stride = tokrows ? (size_t)p.d : (size_t)p.H;
    // Store j of an odd chunk writes column j ^ 1 of the thread's block:
    // wofs[j] is the LDS byte offset of index row idx0 + (j ^ (ch & 1)),
    // chunk ro, and sel_even / sel_odd (for even and odd j) pick the 16-bit
    // halves that form that column.
    const int jx = ch & 1;
    const uint32_t sel_even = jx ? 0x07060302u : 0x05040100u, sel_odd = jx ? 0x05040100u : 0x07060302u;
    uint32_t wofs[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int idx = idx0 + (j ^ jx);
        const int row = isP ? 32 * (idx >> 5) + wcol_pos(idx & 31) : TP + idx;
        wofs[j] = wg_off(row, ro);
    }

    const int nst = (cnt + 63) / 64;
    // Row loads are issued one stage ahead of their LDS store and the list
    // indices two stages ahead, indices first: the memory counter retires in
    // order, so the wait for a stage's indices then never includes the row
    // loads issued after them. No load sits behind a branch (the compiler
    // would then count conservatively): rows past the slab's count read row
    // 0 of the list's buffer and are zeroed before the store, and loads for
    // stages past the last re-read the last one.
    const char* const srcb = reinterpret_cast<const char*>(src);
    const uint32_t row_bytes = (uint32_t)(stride * 2);
    auto load_idx = [&](int st, uint32_t (&ri)[8]) {
        st = min(st, nst - 1);
        const u32x4 a = ld16(list + st * 64), b = ld16(list + st * 64 + 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            ri[q] = a[q];
            ri[4 + q] = b[q];
        }
    };
    auto load_data = [&](int st, const uint32_t (&ri)[8], u32x4 (&v)[8]) {
        st = min(st, nst - 1);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const uint32_t rr = (st * 64 + 8 * ro + q < cnt) ? ri[q] : 0u;
            v[q] = ld16(srcb + (uint64_t)rr * row_bytes);
        }
    };
    auto store_lds = [&](int st, u32x4 (&v)[8]) {
        if (!active) return;
        if (st * 64 + 64 > cnt) {
#pragma unroll
            for (int q = 0; q < 8; ++q)
                if (st * 64 + 8 * ro + q >= cnt) v[q] = u32x4{0u, 0u, 0u, 0u};
        }
        char* base = lds_wg + (st & 1) * STAGE;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            // column j ^ jx: 16-bit half (j ^ jx) & 1 of word j / 2 of the 8 rows
            const uint32_t sel = (j & 1) ? sel_odd : sel_even;
            u32x4 o;
#pragma unroll
            for (int m = 0; m < 4; ++m) o[m] = __builtin_amdgcn_perm(v[2 * m + 1][j >> 1], v[2 * m][j >> 1], sel);
            st16(base + wofs[j], o);
        }
    };
    f32x16 acc[GQ][GP];
#pragma unroll
    for (int i = 0; i < GQ; ++i)
#pragma unroll
        for (int j = 0; j < GP; ++j) acc[i][j] = f32x16{};
    auto compute = [&](int slot) {
        const char* base = lds_wg + slot * STAGE;
#pragma unroll
        for (int kk = 0; kk < S::KSTEPS; ++kk) {
            u32x4 fp[GP], fq[GQ];
#pragma unroll
            for (int j = 0; j < GP; ++j) fp[j] = ld16(base + wg_off(wp * GP * 32 + j * 32 + lr, 2 * kk + lh));
#pragma unroll
            for (int i = 0; i < GQ; ++i) fq[i] = ld16(base + wg_off(TP + wq * GQ * 32 + i * 32 + lr, 2 * kk + lh));
#pragma unroll
            for (int i = 0; i < GQ; ++i)
#pragma unroll
                for (int j = 0; j < GP; ++j) acc[i][j] = mfma32x32x16(as_bf16x8(fp[j]), as_bf16x8(fq[i]), acc[i][j]);
        }
    };
    // Tiles of up to 6 MFMA groups per wave keep two row sets in registers:
    // at stage st the indices of st + 3 and the rows of st + 2 are issued,
    // stage st is multiplied and the rows of st + 1 go to LDS (indices and
    // rows of stage s in set s & 1). Larger tiles keep one row set: the
    // indices of st + 2 and the rows of st + 1 are issued, stage st is
    // multiplied and the rows of st + 1 go to LDS.
    constexpr bool kTwoSets = GQ * GP <= 6;
    uint32_t i0[8], i1[8];
    u32x4 d0[8], d1[8];
    if (nst > 0) {
        load_idx(0, i0);
        load_idx(1, i1);
        load_data(0, i0, d0);
        if constexpr (kTwoSets) {
            load_idx(2, i0);
            load_data(1, i1, d1);
        }
        store_lds(0, d0);
        __syncthreads();
        if constexpr (kTwoSets) {
            auto step = [&](int st, uint32_t (&in)[8], uint32_t (&ic)[8], u32x4 (&dn)[8], u32x4 (&dc)[8]) {
                load_idx(st + 3, in);
                load_data(st + 2, ic, dn);
                compute(st & 1);
                if (st + 1 < nst) store_lds(st + 1, dc);
                __syncthreads();
            };
            int st = 0;
            for (; st + 1 < nst; st += 2) {
                step(st, i1, i0, d0, d1);
                step(st + 1, i0, i1, d1, d0);
            }
            if (st < nst) step(st, i1, i0, d0, d1);
        } else {
            // in: the set of st + 2 (st & 1), ic: the indices of st + 1.
            auto step = [&](int st, uint32_t (&in)[8], uint32_t (&ic)[8]) {
                load_idx(st + 2, in);
                load_data(st + 1, ic, d0);
                compute(st & 1);
                if (st + 1 < nst) store_lds(st + 1, d0);
                __syncthreads();
            };
            int st = 0;
            for (; st + 1 < nst; st += 2) {
                step(st, i0, i1);
                step(st + 1, i1, i0);
            }
            if (st < nst) step(st, i0, i1);
        }
    }
    // Lane: Q index wq GQ 32 + 32 i + lr, P indices wp GP 32 + 32 j + 16 lh + 0..15.
#pragma unroll
    for (int i = 0; i < GQ; ++i) {
        const int qi = wq * GQ * 32 + i * 32 + lr;
        float* row = UP ? p.out + ((size_t)e * p.H + (size_t)c * p.M + qi) * p.d + n0
                        : p.out + ((size_t)e * p.d + n0 + qi) * p.H + (size_t)c * p.M;
#pragma unroll
        for (int j = 0; j < GP; ++j) {
            float* dst = row + wp * GP * 32 + j * 32 + 16 * lh;
            const f32x16 a = acc[i][j];
#pragma unroll
            for (int t = 0; t < 4; ++t)
                st16(dst + 4 * t, u32x4{__float_as_uint(a[4 * t]), __float_as_uint(a[4 * t + 1]),
                                        __float_as_uint(a[4 * t + 2]), __float_as_uint(a[4 * t + 3])});
        }
    }
}

// out[e][j][i] = in[e][i][j] for 16-bit matrices [E][R][C], R and C
// multiples of 64: one 64 x 64 tile per wave; lane (ro, ch) = (lane % 8,
// lane / 8) loads rows 8 ro .. 8 ro + 7 of 16-byte chunk ch and stores the
// transposed 8 x 8 block as 8 rows of 8 (each store instruction writes 8
// whole 128-byte rows).
__global__ __launch_bounds__(256) void transpose16_kernel(const u16* __restrict__ in, u16* __restrict__ out, int R,
                                                           int C, int ntiles) {
    const int t = blockIdx.x * 4 + (int)(threadIdx.x >> 6);
    if (t >= ntiles) return;
    const int tr = R / 64, tc = C / 64;
    const int e = t / (tr * tc), rem = t - e * (tr * tc);
    const int r0 = (rem / tc) * 64, c0 = (rem - (rem / tc) * tc) * 64;
    const int lane = lane_id(), ro = lane & 7, ch = lane >> 3;
    const u16* s = in + (size_t)e * R * C + (size_t)(r0 + 8 * ro) * C + c0 + 8 * ch;
    u32x4 v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = ld16(s + (size_t)q * C);
    u16* d = out + (size_t)e * R * C + (size_t)(c0 + 8 * ch) * R + r0 + 8 * ro;
#pragma unroll
    for (int j = 0; j < 8; ++j) st16(d + (size_t)j * R, column8(v, j));
}

}  // namespace unifmoe
