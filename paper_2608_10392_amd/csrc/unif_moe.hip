// Host side of the UniF-MoE layer library: argument validation, workspace
// planning and the launch sequences. See include/unif_moe.h for the contract
// of every entry point.
//
// Forward launch sequence (all asynchronous on the caller's stream, no
// device-to-host traffic):
//   split_router     fp32 router + prototypes -> 3 bf16 parts (bf16 only);
//                    the same launch clears the counters and tile queues
//   route_logits +   logits with the router held in registers, then the
//   route_decide     decisions, bin slots and per-tile counts (bf16 routers
//                    of at most 32 columns); otherwise one fused route kernel;
//                    extra workgroups of the decisions' launch make the fp16
//                    copy of W_down for the down-projection (bf16 only)
//   scan             segment offsets, bin cursors, per-slab first rows
//   scatter          pairs (expert segments sorted by block-mask key), the
//                    per-(expert, block) row lists in token order and the
//                    up tile table
//   down_tables      down row tiles and their block-mask unions (bf16)
//   up, down         block-sparse MFMA grouped GEMMs              (bf16)
//   pair_ffn_f32     per-pair fp32 FFN                            (fp32)
//   combine          weighted merge in fixed order
// The block forward adds a LayerNorm pass before routing (pre-LN) and
// replaces the merge by the block's merge (biases, residual, post-LN). The
// backward runs routing and the permutation into its workspace, then its
// own kernels (bf16: weight transposes, the x K^T and dy V passes of the up
// engine, the dx pass of the down engine, per-token and router kernels and
// the weight-gradient GEMMs; fp32: vector-unit GEMMs).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "../../include/unif_moe.h"
#include "backward.hpp"
#include "block.hpp"
#include "combine.hpp"
#include "common.hpp"
#include "ffn_bf16.hpp"
#include "ffn_f32.hpp"
#include "permute.hpp"
#include "route.hpp"
#include "stats.hpp"
#include "wgrad.hpp"

using namespace unifmoe;

namespace {

constexpr int kKeyBitsMax = 10;
constexpr int kPhaseEvents = 7;   // unif_moe_layer_forward_profiled
constexpr size_t kLdsLimit = 160 * 1024;

// Expert-GEMM tile shapes, one workgroup of 8 waves per CU. Up: 256 or 384
// gathered rows x the whole block width M. Down: see down_shape.
// Up tiles are 384 rows when the block is at most 192 wide and no stage is
// padding (d >= 256): their accumulators and fragments then still fit two
// waves per SIMD without spills. Else 256.
int up_tm(int M, int d) { return (M <= 192 && d >= 256) ? 384 : 256; }
// Up tiles are ordered by expert, then by groups of blocks, then by the
// stretch of the expert's pairs they cover: the tiles that run together on
// one XCD share token rows (across the group's blocks) and weight slabs
// (within a group). A group's weight slabs take at most this many bytes,
// about 60% of one XCD's 4 MB L2.
constexpr size_t kUpGroupWeightBytes = (size_t)5 << 19;
int up_block_group(int d, int M, int B) {
    const size_t slab = (size_t)2 * d * M;
    return (int)std::max<size_t>(1, std::min<size_t>((size_t)B, kUpGroupWeightBytes / slab));
}
// Down tiles: 256 pairs x 256 columns when d is a multiple of 256, else
// 128 x 384 when d is a multiple of 384 (d = 384: one column tile), else
// 256 x 128.
constexpr int kDownTMMin = 128, kDownTMMax = 256;
constexpr int kDownBNNarrow = 128;
struct DownShape { int tm, bn; };
DownShape down_shape(int d) {
    if (d % 256 == 0) return {256, 256};
    if (d % 384 == 0) return {128, 384};
    return {256, 128};
}
static_assert(up_lds_bytes(192, 384) <= 160 * 1024 && up_lds_bytes(256, 256) <= 160 * 1024, "up stages exceed LDS");
static_assert(down_lds_bytes(128, 384) <= 160 * 1024 && down_lds_bytes(256, 256) <= 160 * 1024,
              "down stages exceed LDS");

struct Dims {
    int N, d, K, B, M, H, K1, NL, NLP, lstride, key_bits, nslab, nbin;
    size_t pcap;   // (token, expert) pairs the forward's workspace holds (cfg max_pairs, else N (K+1))
    bool bf16;
    size_t elem;
    float tau, one_minus_2tau;
};

Dims dims_of(const unif_moe_config* c) {
    Dims m;
    m.N = c->n_tokens;
    m.d = c->d_model;
    m.K = c->n_experts;
    m.B = c->n_blocks;
    m.M = c->block_width;
    m.H = m.B * m.M;
    m.K1 = m.K + 1;
    m.NL = 1 + m.K + m.B;
    m.NLP = ceil_div(m.K + m.B, 16) * 16;   // matrix-core logit rows (bf16 path)
    m.lstride = m.NLP + 1;                  // LDS row: x W_shr, then those
    m.key_bits = m.B < kKeyBitsMax ? m.B : kKeyBitsMax;
    m.nslab = m.K1 * m.B;
    m.nbin = m.K1 << m.key_bits;
    const size_t worst = (size_t)m.N * (size_t)m.K1;
    m.pcap = (c->max_pairs > 0 && (size_t)c->max_pairs < worst) ? (size_t)c->max_pairs : worst;
    m.bf16 = c->dtype == UNIF_BF16;
    m.elem = m.bf16 ? 2 : 4;
    m.tau = std::isnan(c->tau) ? (float)((double)(m.B - 1) / ((double)m.B * (double)m.B)) : c->tau;
    m.one_minus_2tau = 1.0f - 2.0f * m.tau;
    return m;
}

// cfg without a pair capacity (workspaces sized for the worst case).
unif_moe_config worst_case(unif_moe_config c) {
    c.max_pairs = 0;
    return c;
}

// Counters per tile of the permutation: rows per slab, then pairs per expert.
size_t tile_counters(const Dims& m) { return (size_t)m.nslab + m.K1; }
// Routing LDS (route_kernel): the logit rows of its tokens, then its two
// tiles' counters and their tokens' valid flags.
size_t route_lds_bytes(const Dims& m) {
    return sizeof(float) * ((size_t)kRouteTok * m.lstride + (kRouteTok / kTileTok) * (tile_counters(m) + kTileTok));
}
// The persistent logits kernel: 8 partial logit sets of a tile. The
// decisions kernel: a tile's logit rows, counters and valid flags.
size_t route_logits_lds_bytes(const Dims& m) { return sizeof(float) * (size_t)kRpWaves * kRpTok * m.lstride; }
size_t route_decide_lds_bytes(const Dims& m) {
    return sizeof(float) * ((size_t)kTileTok * m.lstride + tile_counters(m) + kTileTok);
}
// Logits of the split routing path (bf16 routers of <= 32 columns, d <= 1024):
// 1 + 16 NCT fp32 values per token, or 0 when the path does not apply.
int split_route_cols(const Dims& m) {
    const int nct = m.NLP / 16, kpw = ceil_div(m.d / 32, kRpWaves);
    return (m.bf16 && nct <= 2 && kpw <= 4) ? 1 + 16 * nct : 0;
}
// The scatter kernel: the tile's tokens' pairs per expert and its first row
// in every slab, or the up tile table's inputs.
size_t scatter_lds_bytes(const Dims& m) {
    const size_t offsets = 2 * ((size_t)m.nslab + 1);
    const size_t token_role = 64 * (size_t)m.K1 + (size_t)m.nslab;
    const size_t table_role = (size_t)kUpTableWords + kScatterWaves * 64 + 64;
    return sizeof(int) * (offsets + std::max(token_role, table_role));
}

// Checks shared by every entry point (host only, no HIP call).
int32_t check_config(const unif_moe_config* c) {
    if (c == nullptr) return UNIF_EINVAL;
    if (c->n_tokens < 0 || c->d_model <= 0 || c->n_experts < 1 || c->n_blocks < 1 || c->block_width < 1)
        return UNIF_EINVAL;
    if (c->max_pairs < 0) return UNIF_EINVAL;
    if (c->dtype != UNIF_F32 && c->dtype != UNIF_BF16) return UNIF_EINVAL;
    if (c->alpha_mode != UNIF_ALPHA_ADAPTIVE && c->alpha_mode != UNIF_ALPHA_FIXED) return UNIF_EINVAL;
    if (c->mass_mode != UNIF_MASS_COUPLED && c->mass_mode != UNIF_MASS_FIXED && c->mass_mode != UNIF_MASS_TOPK)
        return UNIF_EINVAL;
    if (c->select_mode != UNIF_SELECT_PROTOTYPE && c->select_mode != UNIF_SELECT_PREFIX) return UNIF_EINVAL;
    if (!(c->mass_threshold > 0.0f && c->mass_threshold <= 1.0f)) return UNIF_EINVAL;
    if (c->max_shared < 0 || c->max_shared > c->n_blocks) return UNIF_EINVAL;
    if (c->alpha_mode == UNIF_ALPHA_ADAPTIVE && c->n_blocks < 2) return UNIF_EINVAL;
    if (c->alpha_mode == UNIF_ALPHA_FIXED && !(c->alpha_fixed >= 0.0f && c->alpha_fixed <= 1.0f))
        return UNIF_EINVAL;
    if (c->mass_mode == UNIF_MASS_TOPK && (c->fixed_k < 1 || c->fixed_k > c->n_experts)) return UNIF_EINVAL;
    if (!std::isnan(c->tau) && !(c->tau >= 0.0f && c->tau < 0.5f)) return UNIF_EINVAL;
    if (c->n_blocks > 64 || c->n_experts > 64) return UNIF_EUNSUPPORTED;
    const int64_t N = c->n_tokens, K = c->n_experts, B = c->n_blocks;
    if (N * (K + 1) > INT32_MAX || N * K * B > INT32_MAX) return UNIF_EUNSUPPORTED;
    const Dims m = dims_of(c);
    if (route_lds_bytes(m) > kLdsLimit) return UNIF_EUNSUPPORTED;
    if (m.bf16 && (m.d % 32) != 0) return UNIF_EUNSUPPORTED;
    return UNIF_OK;
}

int32_t check_forward_shape(const unif_moe_config* c) {
    const Dims m = dims_of(c);
    if (m.bf16) {
        if (m.d % 128 != 0 || m.M % 64 != 0 || m.M > 256) return UNIF_EUNSUPPORTED;
        // Down tile indices (row tiles x column tiles) fit an int.
        if (((int64_t)m.N * m.K1 / kDownTMMin + m.K1) * (m.d / kDownBNNarrow) >= ((int64_t)1 << 31))
            return UNIF_EUNSUPPORTED;
        if ((int64_t)m.H * m.d * 2 > ((int64_t)1 << 40)) return UNIF_EUNSUPPORTED;
    } else {
        if ((int64_t)m.H > 16384) return UNIF_EUNSUPPORTED;
    }
    return UNIF_OK;
}

// Block description: mode, eps and the shape limit of the post-LN merge
// (checked by the workspace query too).
constexpr int kPostLnMaxD = (int)(kLdsLimit / sizeof(float));   // one fp32 row in LDS
int32_t check_block_shape(const unif_moe_config* c, const unif_moe_block* b) {
    if (b == nullptr) return UNIF_EINVAL;
    if (b->norm != UNIF_NORM_NONE && b->norm != UNIF_NORM_PRE && b->norm != UNIF_NORM_POST) return UNIF_EINVAL;
    if (b->norm != UNIF_NORM_NONE && !(b->ln_eps > 0.0f && std::isfinite(b->ln_eps))) return UNIF_EINVAL;
    if (b->norm == UNIF_NORM_POST && c->d_model > kPostLnMaxD) return UNIF_EUNSUPPORTED;
    return UNIF_OK;
}

// Pointer checks of the block forward.
int32_t check_block_pointers(const unif_moe_config* c, const unif_moe_block* b) {
    if (b->norm != UNIF_NORM_NONE && (b->ln_gamma == nullptr || b->ln_beta == nullptr)) return UNIF_EINVAL;
    // The bf16 kernels read b1 and b2 in 16-byte pieces.
    if (c->dtype == UNIF_BF16 && ((b->b_up != nullptr && reinterpret_cast<uintptr_t>(b->b_up) % 16 != 0) ||
                                  (b->b_down != nullptr && reinterpret_cast<uintptr_t>(b->b_down) % 16 != 0)))
        return UNIF_EINVAL;
    return UNIF_OK;
}

size_t block_xn_bytes(const unif_moe_config* c, const unif_moe_block* b) {
    if (b == nullptr || b->norm != UNIF_NORM_PRE) return 0;
    return (size_t)c->n_tokens * (size_t)c->d_model * (c->dtype == UNIF_BF16 ? 2 : 4);
}

// Workspace carving: regions aligned to 256 bytes.
struct Carver {
    size_t cur = 0;
    size_t take(size_t bytes) {
        cur = (cur + 255) & ~(size_t)255;
        const size_t o = cur;
        cur += bytes;
        return o;
    }
};

struct RoutePlan {
    size_t wsplit, logits, total;
};

RoutePlan plan_route(const Dims& m) {
    Carver cv;
    RoutePlan p;
    p.wsplit = cv.take(m.bf16 ? (size_t)3 * m.NLP * m.d * sizeof(u16) : 0);
    p.logits = cv.take((size_t)m.N * split_route_cols(m) * sizeof(float));
    p.total = cv.cur;
    return p;
}

struct FwdPlan {
    size_t alpha, nsh, mask, nres, eids, wts;
    size_t wsplit, logits;
    size_t zero_begin, zero_end;  // bin_count, slab_count, totals, zero page
    size_t bin_count, slab_count, exp_total, totals, queues, zero_page, work;
    size_t bin_cursor, seg_off, slab_off, down_tile_off, tile_cnt, max_row_tiles, rt_info, rt_masks;
    size_t pair_token, pair_mask, pair_expert, pair_of, pair_rank, slab_rows, slab_tok, up_tile_info, up_tile_rows, hbuf, part;
    size_t xn;      // LN(X), the FFN input of a pre-LN block
    size_t wdown16; // fp16 copy of W_down (bf16 layers)
    size_t down_slices; // [kXcds + 1] down tiles per XCD queue
    size_t total;
};

size_t ceil_div_sz(size_t a, size_t b) { return (a + b - 1) / b; }

// Parts each down tile's block union is split into (the parts' partial rows
// are added by the merge in order). The down kernel runs each tile's blocks
// one after another, so when a workload has no more tiles than a 256-CU
// device has compute units, the chip idles while those chains run: such
// workloads get enough parts for about two tiles per compute unit. The tile
// count is estimated from N with 4 pairs per token (a function of cfg only,
// since it sizes the workspace).
int down_splits(const Dims& m) {
    if (!m.bf16) return 1;
    const DownShape dsh = down_shape(m.d);
    const size_t est_pairs = (size_t)m.N * (size_t)std::min(m.K1, 4);
    const size_t tiles = std::max<size_t>(1, ceil_div_sz(est_pairs, dsh.tm) * (size_t)(m.d / dsh.bn));
    return tiles > 256 ? 1 : (int)std::min<size_t>(4, ceil_div_sz(2 * 256, tiles));
}

// The routing record's region is reserved whether or not the caller passes
// its own record, so every other offset is the same for both kinds of call
// (unif_moe_forward_work reads the workspace a forward left behind).
FwdPlan plan_forward(const Dims& m, size_t xn_bytes = 0) {
    Carver cv;
    FwdPlan p;
    const size_t N = (size_t)m.N, K = (size_t)m.K, K1 = (size_t)m.K1;
    const size_t pmax = m.pcap;   // pairs the pair-indexed buffers hold
    p.alpha = cv.take(4 * N);
    p.nsh = cv.take(4 * N);
    p.mask = cv.take(8 * N);
    p.nres = cv.take(4 * N);
    p.eids = cv.take(4 * N * K);
    p.wts = cv.take(4 * N * K);
    p.wsplit = cv.take(m.bf16 ? (size_t)3 * m.NLP * m.d * sizeof(u16) : 0);
    p.logits = cv.take((size_t)N * split_route_cols(m) * sizeof(float));
    p.bin_count = cv.take(4 * (size_t)m.nbin * kBinCopies);
    p.zero_begin = p.bin_count;
    p.slab_count = cv.take(4 * (size_t)m.nslab);
    p.exp_total = cv.take(4 * (size_t)kExpCopies * K1);
    p.totals = cv.take(4 * 8);
    p.down_slices = cv.take(4 * (kXcds + 1));
    p.queues = cv.take(4 * 16);   // per-XCD tile counters: up, then down
    p.zero_page = cv.take(256);
    p.zero_end = cv.cur;
    p.work = cv.take(16);   // unif_moe_forward_work's counter
    p.bin_cursor = cv.take(4 * (size_t)m.nbin * kBinCopies);
    p.seg_off = cv.take(4 * (K1 + 1));
    p.slab_off = cv.take(4 * ((size_t)m.nslab + 1));
    p.down_tile_off = cv.take(4 * (K1 + 1));
    p.tile_cnt = cv.take(4 * ceil_div_sz(N, kTileTok) * tile_counters(m));
    p.max_row_tiles = ceil_div_sz(pmax, kDownTMMin) + K1;
    p.rt_info = cv.take(m.bf16 ? 16 * p.max_row_tiles : 0);
    p.rt_masks = cv.take(m.bf16 ? 8 * (kDownTMMax / 32 + 1) * p.max_row_tiles : 0);
    p.pair_token = cv.take(4 * pmax);
    p.pair_mask = cv.take(8 * (pmax + kDownTMMax));   // a whole down tile is readable past the last pair
    p.pair_expert = cv.take(4 * pmax);
    p.pair_of = cv.take(4 * N * K1);
    p.pair_rank = cv.take(4 * N * K1);
    // Slab row lists: at most K B rows per token (b + k (B - b) <= K B) and
    // at most B per pair, each slab padded to whole up tiles.
    const size_t tm = (size_t)up_tm(m.M, m.d);
    const size_t up_tiles = ceil_div_sz(std::min(N * K, pmax) * (size_t)m.B, tm) + (size_t)m.nslab;
    p.slab_rows = cv.take(m.bf16 ? 4 * up_tiles * tm : 0);
    p.slab_tok = cv.take(m.bf16 ? 4 * up_tiles * tm : 0);
    p.up_tile_info = cv.take(m.bf16 ? 4 * up_tiles : 0);
    p.up_tile_rows = cv.take(m.bf16 ? 4 * up_tiles : 0);
    p.hbuf = cv.take(m.bf16 ? (pmax + 1) * (size_t)m.H * 2 : 0);  // fp16, + the sink row
    p.part = cv.take((pmax + 1) * (size_t)m.d * sizeof(float) * down_splits(m));   // fp32, + the sink row, per part
    p.xn = cv.take(xn_bytes);
    p.wdown16 = cv.take(m.bf16 ? K1 * (size_t)m.d * m.H * 2 : 0);
    p.total = cv.cur + 256;  // slack for aligning an unaligned base pointer
    return p;
}

char* align_base(void* ws) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(ws);
    return reinterpret_cast<char*>((a + 255) & ~(uintptr_t)255);
}

// Compute units of the current device (queried at each call; the grids of
// the persistent kernels are sized by it).
int cu_count() {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
    return n;
}

#define UNIF_LAUNCH_CHECK()                              \
    do {                                                 \
        if (hipGetLastError() != hipSuccess) return UNIF_EDEVICE; \
    } while (0)

template <class F>
int32_t allow_lds(F* kernel, size_t bytes) {
    if (bytes <= 64 * 1024) return UNIF_OK;
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)bytes) != hipSuccess)
        return UNIF_EDEVICE;
    return UNIF_OK;
}

template <class P>
int32_t launch_persistent(void (*kernel)(P), int grid, size_t lds, hipStream_t st, const P& prm) {
    if (allow_lds(kernel, lds) != UNIF_OK) return UNIF_EDEVICE;
    kernel<<<grid, kFfnThreads, lds, st>>>(prm);
    return hipGetLastError() == hipSuccess ? UNIF_OK : UNIF_EDEVICE;
}

RouteParams route_params(const unif_moe_config* c, const Dims& m, const void* X, const uint8_t* valid,
                         const float* Wr, const float* mu, const u16* wsplit, float* alpha, int* nsh,
                         uint64_t* mask, int* nres, int* eids, float* wts) {
    RouteParams r;
    r.N = m.N;
    r.d = m.d;
    r.K = m.K;
    r.B = m.B;
    r.NL = m.NL;
    r.NLP = m.NLP;
    r.lstride = m.lstride;
    r.key_bits = m.key_bits;
    r.tau = m.tau;
    r.one_minus_2tau = m.one_minus_2tau;
    r.t_mass = c->mass_threshold;
    r.alpha_fixed = c->alpha_fixed;
    r.max_shared = c->max_shared;
    r.alpha_mode = c->alpha_mode;
    r.mass_mode = c->mass_mode;
    r.fixed_k = c->fixed_k;
    r.select_mode = c->select_mode;
    r.X = X;
    r.valid = valid;
    r.Wr = Wr;
    r.mu = mu;
    r.Wsplit = wsplit;
    r.alpha = alpha;
    r.nsh = nsh;
    r.mask = mask;
    r.nres = nres;
    r.eids = eids;
    r.wts = wts;
    r.bin_count = nullptr;
    r.tile_cnt = nullptr;
    r.exp_total = nullptr;
    r.pair_rank = nullptr;
    r.cvt_src = nullptr;
    r.cvt_dst = nullptr;
    r.cvt_n8 = 0;
    r.cvt_blocks = 0;
    return r;
}

// Router logits and decisions (shared by unif_moe_route and the forward).
// The forward's counters (zwords words at zero) are cleared in the launch
// that splits the router weights.
int32_t launch_route(const Dims& m, const RouteParams& rp, const float* Wr, const float* mu, u16* wsplit,
                     float* logits, hipStream_t st, uint32_t* zero = nullptr, size_t zwords = 0) {
    if (m.N == 0) return UNIF_OK;
    const int nsplit = m.bf16 ? ceil_div(m.NLP * m.d, 256) : 0;
    const int nzero = zwords ? (int)std::min<size_t>(ceil_div_sz(zwords, 256), 1024) : 0;
    if (nsplit + nzero > 0) {
        split_router_kernel<<<nsplit + nzero, 256, 0, st>>>(Wr, mu, m.K, m.B, m.d, m.NLP, wsplit, nsplit, zero,
                                                           zwords);
        UNIF_LAUNCH_CHECK();
    }
    // Small bf16 routers: logits (router in registers), then decisions.
    const int ncols = split_route_cols(m);
    if (ncols > 0 && logits != nullptr) {
        void (*lk)(RouteParams, float*) = nullptr;
        const int nct = m.NLP / 16, kpw = ceil_div(m.d / 32, kRpWaves);
        switch (nct * 4 + kpw) {
            case 5: lk = route_logits_kernel<1, 1>; break;
            case 6: lk = route_logits_kernel<1, 2>; break;
            case 7: lk = route_logits_kernel<1, 3>; break;
            case 9: lk = route_logits_kernel<2, 1>; break;
            case 10: lk = route_logits_kernel<2, 2>; break;
            case 11: lk = route_logits_kernel<2, 3>; break;
            case 8: lk = route_logits_kernel<1, 4>; break;
            case 12: lk = route_logits_kernel<2, 4>; break;
            default: return UNIF_EUNSUPPORTED;
        }
        void (*dk)(RouteParams, const float*, int) = nullptr;
        const int ntiles = ceil_div(m.N, kRpTok);
        const bool wide = ntiles <= 2 * cu_count();   // 8 waves per tile
        switch (decide_lanes(m.K, m.B)) {
            case 16: dk = wide ? route_decide_kernel<16, 8> : route_decide_kernel<16, 4>; break;
            case 32: dk = wide ? route_decide_kernel<32, 8> : route_decide_kernel<32, 4>; break;
            default: dk = wide ? route_decide_kernel<64, 8> : route_decide_kernel<64, 4>; break;
        }
        const size_t l1 = route_logits_lds_bytes(m), l2 = route_decide_lds_bytes(m);
        if (allow_lds(lk, l1) != UNIF_OK || allow_lds(dk, l2) != UNIF_OK) return UNIF_EDEVICE;
        lk<<<std::min(cu_count(), ntiles), kRpThreads, l1, st>>>(rp, logits);
        UNIF_LAUNCH_CHECK();
        dk<<<ntiles + rp.cvt_blocks, wide ? 512 : 256, l2, st>>>(rp, logits, ncols);
        UNIF_LAUNCH_CHECK();
        return UNIF_OK;
    }
    const size_t lds = route_lds_bytes(m);
    const int grid = ceil_div(m.N, kRouteTok);
    void (*kern)(RouteParams) = route_kernel<0>;
    if (m.bf16) {
        switch (m.NLP / 16) {
            case 1: kern = route_kernel<1>; break;
            case 2: kern = route_kernel<2>; break;
            case 3: kern = route_kernel<3>; break;
            case 4: kern = route_kernel<4>; break;
            case 5: kern = route_kernel<5>; break;
            case 6: kern = route_kernel<6>; break;
            case 7: kern = route_kernel<7>; break;
            case 8: kern = route_kernel<8>; break;
            default: return UNIF_EUNSUPPORTED;
        }
    }
    if (allow_lds(kern, lds) != UNIF_OK) return UNIF_EDEVICE;
    kern<<<grid + rp.cvt_blocks, kRouteThreads, lds, st>>>(rp);
    UNIF_LAUNCH_CHECK();
    return UNIF_OK;
}

bool record_complete(const unif_moe_routing* r) {
    return r && r->alpha && r->n_shared && r->shared_mask && r->n_res && r->expert_ids && r->weights;
}

}  // namespace

extern "C" {

const char* unif_moe_status_string(int32_t s) {
    switch (s) {
        case UNIF_OK: return "ok";
        case UNIF_EINVAL: return "invalid argument";
        case UNIF_EWORKSPACE: return "workspace too small";
        case UNIF_EDEVICE: return "HIP device error";
        case UNIF_EUNSUPPORTED: return "unsupported layer shape";
        case UNIF_ECAPACITY: return "routing needs more pairs than the capacity";
        default: return "unknown status";
    }
}

int32_t unif_moe_route_workspace_size(const unif_moe_config* cfg, size_t* bytes) {
    if (bytes == nullptr) return UNIF_EINVAL;
    const int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    const RoutePlan p = plan_route(dims_of(cfg));
    *bytes = p.total ? p.total + 256 : 0;
    return UNIF_OK;
}

int32_t unif_moe_route(const unif_moe_config* cfg, const void* X, const uint8_t* valid, const float* W_router,
                       const float* prototypes, const unif_moe_routing* out, void* workspace,
                       size_t workspace_bytes, void* stream) {
    int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    if (!record_complete(out)) return UNIF_EINVAL;
    if (cfg->n_tokens > 0 && (X == nullptr || W_router == nullptr || prototypes == nullptr)) return UNIF_EINVAL;
    size_t need = 0;
    unif_moe_route_workspace_size(cfg, &need);
    if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return UNIF_EWORKSPACE;
    const Dims m = dims_of(cfg);
    const RoutePlan plan = plan_route(m);
    char* ws = need ? align_base(workspace) : nullptr;
    u16* wsplit = m.bf16 ? reinterpret_cast<u16*>(ws + plan.wsplit) : nullptr;
    const RouteParams rp = route_params(cfg, m, X, valid, W_router, prototypes, wsplit, out->alpha,
                                        out->n_shared, out->shared_mask, out->n_res, out->expert_ids,
                                        out->weights);
    float* logits = need ? reinterpret_cast<float*>(ws + plan.logits) : nullptr;
    return launch_route(m, rp, W_router, prototypes, wsplit, logits, static_cast<hipStream_t>(stream));
}

int32_t unif_moe_layer_forward_workspace_size(const unif_moe_config* cfg, size_t* bytes) {
    if (bytes == nullptr) return UNIF_EINVAL;
    int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    s = check_forward_shape(cfg);
    if (s != UNIF_OK) return s;
    *bytes = plan_forward(dims_of(cfg)).total;
    return UNIF_OK;
}

}  // extern "C"

namespace {

int32_t record_event(void* const* events, int i, hipStream_t st) {
    if (events == nullptr) return UNIF_OK;
    return hipEventRecord(static_cast<hipEvent_t>(events[i]), st) == hipSuccess ? UNIF_OK : UNIF_EDEVICE;
}

#define UNIF_MARK(i)                                        \
    do {                                                    \
        if (record_event(events, (i), st) != UNIF_OK) return UNIF_EDEVICE; \
    } while (0)

// Up-projection launch for the layer's block width, with epilogue EPI.
template <int EPI>
int32_t launch_up(const Dims& m, int grid, size_t lds, hipStream_t st, const UpParams& up) {
    const bool pad = m.d < 256;
    switch (m.M / 64) {
        case 1:
            return pad ? launch_persistent(up_kernel<1, true, 256, EPI>, grid, lds, st, up)
                       : launch_persistent(up_kernel<1, false, 384, EPI>, grid, lds, st, up);
        case 2:
            return pad ? launch_persistent(up_kernel<2, true, 256, EPI>, grid, lds, st, up)
                       : launch_persistent(up_kernel<2, false, 384, EPI>, grid, lds, st, up);
        case 3:
            return pad ? launch_persistent(up_kernel<3, true, 256, EPI>, grid, lds, st, up)
                       : launch_persistent(up_kernel<3, false, 384, EPI>, grid, lds, st, up);
        case 4:
            return pad ? launch_persistent(up_kernel<4, true, 256, EPI>, grid, lds, st, up)
                       : launch_persistent(up_kernel<4, false, 256, EPI>, grid, lds, st, up);
        default: return UNIF_EUNSUPPORTED;
    }
}

// The layer forward (blk == nullptr) or the block forward around it.
int32_t forward_impl(const unif_moe_config* cfg, const unif_moe_block* blk, const void* X,
                     const uint8_t* valid, const float* W_router, const float* prototypes,
                     const void* W_up, const void* W_down, void* Y,
                     const unif_moe_routing* routing_out, void* workspace, size_t workspace_bytes,
                     void* const* events, void* stream, bool tables_only = false) {
    int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    s = check_forward_shape(cfg);
    if (s != UNIF_OK) return s;
    if (blk != nullptr) {
        s = check_block_shape(cfg, blk);
        if (s != UNIF_OK) return s;
        s = check_block_pointers(cfg, blk);
        if (s != UNIF_OK) return s;
    }
    if (routing_out != nullptr && !record_complete(routing_out)) return UNIF_EINVAL;
    if (cfg->n_tokens > 0 && (X == nullptr || W_router == nullptr || prototypes == nullptr ||
                              W_up == nullptr || W_down == nullptr || (Y == nullptr && !tables_only)))
        return UNIF_EINVAL;
    const Dims m = dims_of(cfg);
    const bool own = routing_out == nullptr;
    const FwdPlan plan = plan_forward(m, block_xn_bytes(cfg, blk));
    // The size reported by the query always includes the internal record.
    size_t need = 0;
    if (blk != nullptr) unif_moe_block_forward_workspace_size(cfg, blk, &need);
    else unif_moe_layer_forward_workspace_size(cfg, &need);
    if (workspace == nullptr || workspace_bytes < need) return UNIF_EWORKSPACE;
    if (m.N == 0) return UNIF_OK;

    hipStream_t st = static_cast<hipStream_t>(stream);
    char* ws = align_base(workspace);
    float* alpha = own ? reinterpret_cast<float*>(ws + plan.alpha) : routing_out->alpha;
    int* nsh = own ? reinterpret_cast<int*>(ws + plan.nsh) : routing_out->n_shared;
    uint64_t* mask = own ? reinterpret_cast<uint64_t*>(ws + plan.mask) : routing_out->shared_mask;
    int* nres = own ? reinterpret_cast<int*>(ws + plan.nres) : routing_out->n_res;
    int* eids = own ? reinterpret_cast<int*>(ws + plan.eids) : routing_out->expert_ids;
    float* wts = own ? reinterpret_cast<float*>(ws + plan.wts) : routing_out->weights;
    u16* wsplit = m.bf16 ? reinterpret_cast<u16*>(ws + plan.wsplit) : nullptr;
    int* bin_count = reinterpret_cast<int*>(ws + plan.bin_count);
    int* slab_count = reinterpret_cast<int*>(ws + plan.slab_count);
    int* totals = reinterpret_cast<int*>(ws + plan.totals);

    UNIF_MARK(0);
    // 0. the fp16 copy of W_down that the down-projection multiplies with:
    // made by extra workgroups of the routing decisions' launch (step 2)
    const u16* wdown16 = (m.bf16 && !tables_only) ? reinterpret_cast<u16*>(ws + plan.wdown16) : nullptr;
    UNIF_MARK(1);
    // 1. the FFN input: LN(X) for a pre-LN block, else X
    const void* Xf = X;
    if (blk != nullptr && blk->norm == UNIF_NORM_PRE) {
        LayerNormParams ln;
        ln.N = m.N;
        ln.d = m.d;
        ln.X = X;
        ln.Xn = ws + plan.xn;
        ln.gamma = blk->ln_gamma;
        ln.beta = blk->ln_beta;
        ln.eps = (double)blk->ln_eps;
        // 16 lanes per row, 16 rows per workgroup; rows of up to 1024 bf16
        // (128 fp32) stay in registers.
        const unsigned g = (unsigned)ceil_div(m.N, 16);
        if (m.bf16) layernorm_rows_kernel<true, 8, 16><<<g, 256, 0, st>>>(ln);
        else layernorm_rows_kernel<false, 8, 16><<<g, 256, 0, st>>>(ln);
        UNIF_LAUNCH_CHECK();
        Xf = ln.Xn;
    }
    // 1. zero the counters (in the launch before routing) and 2. routing + counts
    const size_t zwords = (plan.zero_end - plan.zero_begin) / 4;
    RouteParams rp = route_params(cfg, m, Xf, valid, W_router, prototypes, wsplit, alpha, nsh, mask, nres, eids,
                                  wts);
    rp.bin_count = bin_count;
    rp.tile_cnt = reinterpret_cast<int*>(ws + plan.tile_cnt);
    rp.exp_total = reinterpret_cast<int*>(ws + plan.exp_total);
    rp.pair_rank = reinterpret_cast<int*>(ws + plan.pair_rank);
    if (wdown16 != nullptr) {
        rp.cvt_src = static_cast<const u16*>(W_down);
        rp.cvt_dst = reinterpret_cast<u16*>(ws + plan.wdown16);
        rp.cvt_n8 = (size_t)m.K1 * m.d * m.H / 8;
        rp.cvt_blocks = (int)std::min<size_t>(ceil_div_sz(rp.cvt_n8, 256), (size_t)cu_count() * 2);
    }
    s = launch_route(m, rp, W_router, prototypes, wsplit, reinterpret_cast<float*>(ws + plan.logits), st,
                     reinterpret_cast<uint32_t*>(ws + plan.zero_begin), zwords);
    if (s != UNIF_OK) return s;
    UNIF_MARK(2);

    // 3. offsets and tile tables, pair slots, slab lists
    PermuteParams pp;
    pp.N = m.N;
    pp.K = m.K;
    pp.B = m.B;
    pp.key_bits = m.key_bits;
    const DownShape dsh = down_shape(m.d);
    pp.bm_up = up_tm(m.M, m.d);
    pp.up_group = up_block_group(m.d, m.M, m.B);
    pp.bm_down = dsh.tm;
    pp.down_col_tiles = m.bf16 ? m.d / dsh.bn : 1;
    pp.mask = mask;
    pp.nres = nres;
    pp.eids = eids;
    pp.bin_count = bin_count;
    pp.bin_cursor = reinterpret_cast<int*>(ws + plan.bin_cursor);
    pp.slab_count = slab_count;
    pp.slab_off = reinterpret_cast<int*>(ws + plan.slab_off);
    pp.seg_off = reinterpret_cast<int*>(ws + plan.seg_off);
    pp.down_tile_off = reinterpret_cast<int*>(ws + plan.down_tile_off);
    pp.totals = totals;
    pp.pair_token = reinterpret_cast<int*>(ws + plan.pair_token);
    pp.pair_mask = reinterpret_cast<uint64_t*>(ws + plan.pair_mask);
    pp.pair_expert = reinterpret_cast<int*>(ws + plan.pair_expert);
    pp.pair_of = reinterpret_cast<int*>(ws + plan.pair_of);
    pp.slab_rows = m.bf16 ? reinterpret_cast<int*>(ws + plan.slab_rows) : nullptr;
    pp.slab_tok = m.bf16 ? reinterpret_cast<int*>(ws + plan.slab_tok) : nullptr;
    pp.up_tile_info = m.bf16 ? reinterpret_cast<int*>(ws + plan.up_tile_info) : nullptr;
    pp.up_tile_rows = m.bf16 ? reinterpret_cast<int*>(ws + plan.up_tile_rows) : nullptr;
    pp.tile_cnt = reinterpret_cast<int*>(ws + plan.tile_cnt);
    pp.exp_total = rp.exp_total;
    pp.rt_info = m.bf16 ? reinterpret_cast<int4*>(ws + plan.rt_info) : nullptr;
    pp.rt_masks = m.bf16 ? reinterpret_cast<uint64_t*>(ws + plan.rt_masks) : nullptr;
    pp.pair_rank = rp.pair_rank;
    pp.ntile = ceil_div(m.N, kTileTok);
    pp.max_pairs = (int)m.pcap;
    pp.down_slices = reinterpret_cast<int*>(ws + plan.down_slices);
    pp.down_stages = m.M / 64;
    // The backward (tables_only) runs its down-projection unsplit.
    pp.down_splits = tables_only ? 1 : down_splits(m);
    // Expert segments and bin cursors; per slab (bf16), its rows per token
    // tile as first rows.
    scan_kernel<<<(unsigned)(m.K1 + (m.bf16 ? m.nslab : 0)), kScanThreads, 0, st>>>(pp);
    UNIF_LAUNCH_CHECK();
    // Pairs and slab rows; the up tile table (bf16).
    const int up_groups = m.bf16 ? m.K1 * ceil_div(m.B, pp.up_group) : 0;
    {
        const size_t lds = scatter_lds_bytes(m);
        if (allow_lds(scatter_kernel, lds) != UNIF_OK) return UNIF_EDEVICE;
        scatter_kernel<<<(unsigned)(up_groups + pp.ntile), kScatterWaves * 64, lds, st>>>(
            pp, up_groups);
        UNIF_LAUNCH_CHECK();
    }

    const int cus = cu_count();
    void* part = ws + plan.part;
    if (m.bf16) {
        // Down row-tile descriptions (the grid-stride loop is sized for the
        // worst case only up to a few workgroups per CU).
        down_tables_kernel<<<(unsigned)std::min<size_t>(ceil_div_sz(plan.max_row_tiles, 4), (size_t)cus * 4), 256, 0,
                             st>>>(pp);
        UNIF_LAUNCH_CHECK();
        // The down tiles of each XCD's queue, split by cost.
        down_slices_kernel<<<1, kSliceThreads, 0, st>>>(pp);
        UNIF_LAUNCH_CHECK();
        UNIF_MARK(3);
        if (tables_only) return UNIF_OK;
        // 4. block-sparse expert GEMMs
        UpParams up;
        up.d = m.d;
        up.M = m.M;
        up.B = m.B;
        up.H = m.H;
        up.X = static_cast<const u16*>(Xf);
        up.Wup = static_cast<const u16*>(W_up);
        up.Hbuf = reinterpret_cast<u16*>(ws + plan.hbuf);
        up.Hsink = up.Hbuf + m.pcap * m.H;
        up.sink_row = m.pcap;
        up.Gbuf = nullptr;
        up.pw = nullptr;
        up.dcp = nullptr;
        up.slab_rows = pp.slab_rows;
        up.slab_tok = pp.slab_tok;
        up.tile_info = pp.up_tile_info;
        up.tile_rows = pp.up_tile_rows;
        up.totals = totals;
        up.queue = reinterpret_cast<int*>(ws + plan.queues);
        up.b_up = blk != nullptr ? blk->b_up : nullptr;
        const size_t up_lds = (size_t)up_lds_bytes(m.M, up_tm(m.M, m.d));
        const int grid = (cus / kXcds) * kXcds;
        s = up.b_up != nullptr ? launch_up<kEpiGeluBias>(m, grid, up_lds, st, up)
                                : launch_up<kEpiGelu>(m, grid, up_lds, st, up);
        if (s != UNIF_OK) return s;
        UNIF_MARK(4);
        DownParams dn;
        dn.d = m.d;
        dn.M = m.M;
        dn.B = m.B;
        dn.H = m.H;
        dn.ncol = pp.down_col_tiles;
        dn.zero16 = reinterpret_cast<const u16*>(ws + plan.zero_page);
        dn.Hbuf = up.Hbuf;
        dn.Wdown = wdown16;
        dn.part = static_cast<float*>(part);
        dn.part_sink = dn.part + m.pcap * m.d;
        dn.rt_info = pp.rt_info;
        dn.rt_masks = pp.rt_masks;
        dn.pair_mask = pp.pair_mask;
        dn.slices = pp.down_slices;
        dn.queue = reinterpret_cast<int*>(ws + plan.queues) + 8;
        dn.nsplit = down_splits(m);
        dn.split_stride = (m.pcap + 1) * m.d;
        if (dsh.bn == 384)
            s = launch_persistent(down_kernel<2, 3>, grid, (size_t)down_lds_bytes(128, 384), st, dn);
        else if (dsh.bn == 256)
            s = launch_persistent(down_kernel<4, 4>, grid, (size_t)down_lds_bytes(256, 256), st, dn);
        else
            s = launch_persistent(down_kernel<4, 2>, grid, (size_t)down_lds_bytes(256, 128), st, dn);
        if (s != UNIF_OK) return s;
        UNIF_MARK(5);
    } else {
        UNIF_MARK(3);
        if (tables_only) return UNIF_OK;
        PairF32Params fp;
        fp.d = m.d;
        fp.M = m.M;
        fp.B = m.B;
        fp.H = m.H;
        fp.X = static_cast<const float*>(Xf);
        fp.b_up = blk != nullptr ? blk->b_up : nullptr;
        fp.Wup = static_cast<const float*>(W_up);
        fp.Wdown = static_cast<const float*>(W_down);
        fp.part = static_cast<float*>(part);
        fp.pair_token = pp.pair_token;
        fp.pair_expert = pp.pair_expert;
        fp.pair_mask = pp.pair_mask;
        fp.totals = totals;
        const size_t lds = (size_t)m.H * sizeof(float);
        if (allow_lds(pair_ffn_f32_kernel, lds) != UNIF_OK) return UNIF_EDEVICE;
        pair_ffn_f32_kernel<<<cus * 4, 256, lds, st>>>(fp);
        UNIF_LAUNCH_CHECK();
        UNIF_MARK(4);
        UNIF_MARK(5);
    }

    // 5. weighted merge (the block's merge around it)
    if (blk != nullptr) {
        BlockCombineParams bc;
        bc.nsplit = down_splits(m);
        bc.split_stride = (m.pcap + 1) * m.d;
        bc.N = m.N;
        bc.d = m.d;
        bc.K = m.K;
        bc.B = m.B;
        bc.part = part;
        bc.pair_of = pp.pair_of;
        bc.alpha = alpha;
        bc.nsh = nsh;
        bc.nres = nres;
        bc.eids = eids;
        bc.wts = wts;
        bc.b_down = blk->b_down;
        bc.X = blk->residual ? X : nullptr;
        bc.post = blk->norm == UNIF_NORM_POST;
        bc.gamma = blk->ln_gamma;
        bc.beta = blk->ln_beta;
        bc.eps = (double)blk->ln_eps;
        bc.Y = Y;
        bc.totals = totals;
        if (!bc.post) {
            const int nch = m.bf16 ? m.d / 8 : m.d;
            const unsigned g = (unsigned)(((size_t)m.N * nch + 255) / 256);
            if (m.bf16) combine_block_flat_kernel<true><<<g, 256, 0, st>>>(bc);
            else combine_block_flat_kernel<false><<<g, 256, 0, st>>>(bc);
        } else {
            // One fp32 row per wave in LDS: 4 rows per workgroup while that
            // fits in 64 KB, else one.
            const int rows = ((size_t)16 * m.d <= 65536) ? 4 : 1;
            const size_t lds = (size_t)rows * m.d * sizeof(float);
            const unsigned g = (unsigned)ceil_div(m.N, rows);
            if (m.bf16) {
                if (allow_lds(combine_block_post_kernel<true>, lds) != UNIF_OK) return UNIF_EDEVICE;
                combine_block_post_kernel<true><<<g, 64 * rows, lds, st>>>(bc);
            } else {
                if (allow_lds(combine_block_post_kernel<false>, lds) != UNIF_OK) return UNIF_EDEVICE;
                combine_block_post_kernel<false><<<g, 64 * rows, lds, st>>>(bc);
            }
        }
        UNIF_LAUNCH_CHECK();
        UNIF_MARK(6);
        return UNIF_OK;
    }
    CombineParams cp;
    cp.nsplit = down_splits(m);
    cp.split_stride = (m.pcap + 1) * m.d;
    cp.N = m.N;
    cp.d = m.d;
    cp.K = m.K;
    cp.part = part;
    cp.pair_of = pp.pair_of;
    cp.alpha = alpha;
    cp.nres = nres;
    cp.wts = wts;
    cp.Y = Y;
    cp.totals = totals;
    if (m.bf16) {
        const size_t items = (size_t)m.N * (m.d / 4);
        if (cp.nsplit > 1) combine_bf16_kernel<true><<<(unsigned)((items + 255) / 256), 256, 0, st>>>(cp);
        else combine_bf16_kernel<false><<<(unsigned)((items + 255) / 256), 256, 0, st>>>(cp);
    } else {
        const size_t items = (size_t)m.N * m.d;
        combine_f32_kernel<<<(unsigned)((items + 255) / 256), 256, 0, st>>>(cp);
    }
    UNIF_LAUNCH_CHECK();
    UNIF_MARK(6);
    return UNIF_OK;
}

}  // namespace

extern "C" {

int32_t unif_moe_layer_forward(const unif_moe_config* cfg, const void* X, const uint8_t* valid,
                               const float* W_router, const float* prototypes, const void* W_up,
                               const void* W_down, void* Y, const unif_moe_routing* routing_out,
                               void* workspace, size_t workspace_bytes, void* stream) {
    return forward_impl(cfg, nullptr, X, valid, W_router, prototypes, W_up, W_down, Y, routing_out,
                        workspace, workspace_bytes, nullptr, stream);
}

int32_t unif_moe_block_forward_workspace_size(const unif_moe_config* cfg, const unif_moe_block* blk,
                                              size_t* bytes) {
    if (bytes == nullptr) return UNIF_EINVAL;
    int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    s = check_forward_shape(cfg);
    if (s != UNIF_OK) return s;
    s = check_block_shape(cfg, blk);
    if (s != UNIF_OK) return s;
    *bytes = plan_forward(dims_of(cfg), block_xn_bytes(cfg, blk)).total;
    return UNIF_OK;
}

int32_t unif_moe_block_forward(const unif_moe_config* cfg, const unif_moe_block* blk, const void* X,
                               const uint8_t* valid, const float* W_router, const float* prototypes,
                               const void* W_up, const void* W_down, void* Y,
                               const unif_moe_routing* routing_out, void* workspace, size_t workspace_bytes,
                               void* stream) {
    if (blk == nullptr) return UNIF_EINVAL;
    return forward_impl(cfg, blk, X, valid, W_router, prototypes, W_up, W_down, Y, routing_out, workspace,
                        workspace_bytes, nullptr, stream);
}

int32_t unif_moe_layer_forward_profiled(const unif_moe_config* cfg, const void* X, const uint8_t* valid,
                                        const float* W_router, const float* prototypes, const void* W_up,
                                        const void* W_down, void* Y, const unif_moe_routing* routing_out,
                                        void* workspace, size_t workspace_bytes, void* const* events,
                                        int32_t n_events, void* stream) {
    if (events == nullptr || n_events != kPhaseEvents) return UNIF_EINVAL;
    for (int i = 0; i < kPhaseEvents; ++i)
        if (events[i] == nullptr) return UNIF_EINVAL;
    return forward_impl(cfg, nullptr, X, valid, W_router, prototypes, W_up, W_down, Y, routing_out, workspace,
                        workspace_bytes, events, stream);
}

}  // extern "C"

namespace {

// Backward workspace: the forward's (routing record, pair tables, slab
// lists; for bf16 layers its H buffer holds GELU(a), then w GELU(a), and its
// fp16 W_down region the transposed W_up; its per-pair rows receive dx_pair),
// then for bf16 layers a second H-shaped buffer (GELU'(a), then d loss / da),
// V^T and the per-(pair, block) partial sums of dy . E, for fp32 layers the
// per-pair fp32 intermediates, and the per-pair and per-token scalars.
struct BwdPlan {
    size_t fwd, act, da, gbuf, wdnT, dcp, dcoef, pw, dz, rpart, queues, total;
};

BwdPlan plan_backward(const Dims& m) {
    BwdPlan b;
    b.fwd = plan_forward(m).total;   // includes its own 256 bytes of alignment slack
    const size_t pmax = (size_t)m.N * m.K1;
    Carver cv;
    cv.cur = b.fwd;
    b.act = cv.take(m.bf16 ? 0 : pmax * m.H * sizeof(float));
    b.da = cv.take(m.bf16 ? 0 : pmax * m.H * sizeof(float));
    b.gbuf = cv.take(m.bf16 ? (pmax + 1) * (size_t)m.H * 2 : 0);   // + the sink row
    b.wdnT = cv.take(m.bf16 ? (size_t)m.K1 * m.d * m.H * 2 : 0);
    b.dcp = cv.take(m.bf16 ? (pmax + 1) * m.B * 2 * sizeof(float) : 0);
    b.dcoef = cv.take(pmax * sizeof(float));
    b.pw = cv.take(pmax * sizeof(float));
    b.dz = cv.take((size_t)m.N * m.K1 * sizeof(float));
    b.rpart = cv.take((size_t)kRouterChunks * m.K1 * m.d * sizeof(float));
    b.queues = cv.take(4 * 32);
    b.total = cv.cur + 256;
    return b;
}

int32_t check_backward_shape(const unif_moe_config* c) {
    int32_t s = check_config(c);
    if (s != UNIF_OK) return s;
    s = check_forward_shape(c);
    if (s != UNIF_OK) return s;
    // fp32 layers: pair tiles of an expert segment index grid dimension y.
    if (c->dtype == UNIF_F32 && ceil_div(c->n_tokens, kBT) > 65535) return UNIF_EUNSUPPORTED;
    // the per-token and router-gradient kernels take 4 and 8 columns at a time
    if (c->d_model % 8 != 0) return UNIF_EUNSUPPORTED;
    return UNIF_OK;
}

// The weight-gradient launch for block width M and n tiles of TN columns.
template <bool UP, int GQ, int GP, int WQ>
int32_t launch_wgrad1(const WgradParams& w, int nslab, hipStream_t st) {
    constexpr int TQ = WQ * GQ * 32, TP = (8 / WQ) * GP * 32;
    const size_t lds = (size_t)wgrad_lds_bytes(TQ, TP);
    if (allow_lds(wgrad_kernel<UP, GQ, GP, WQ>, lds) != UNIF_OK) return UNIF_EDEVICE;
    wgrad_kernel<UP, GQ, GP, WQ><<<(unsigned)(nslab * w.ntn), 512, lds, st>>>(w);
    return hipGetLastError() == hipSuccess ? UNIF_OK : UNIF_EDEVICE;
}

template <bool UP, int GN>
int32_t launch_wgrad_m(const WgradParams& w, int nslab, hipStream_t st) {
    // dW_up: Q = h (2 waves x M / 64 groups), P = n (4 waves x GN groups);
    // dW_down: Q = n (4 waves x GN groups), P = h (2 waves x M / 64 groups).
    switch (w.M / 64) {
        case 1: return UP ? launch_wgrad1<true, 1, GN, 2>(w, nslab, st) : launch_wgrad1<false, GN, 1, 4>(w, nslab, st);
        case 2: return UP ? launch_wgrad1<true, 2, GN, 2>(w, nslab, st) : launch_wgrad1<false, GN, 2, 4>(w, nslab, st);
        case 3: return UP ? launch_wgrad1<true, 3, GN, 2>(w, nslab, st) : launch_wgrad1<false, GN, 3, 4>(w, nslab, st);
        case 4: return UP ? launch_wgrad1<true, 4, GN, 2>(w, nslab, st) : launch_wgrad1<false, GN, 4, 4>(w, nslab, st);
        default: return UNIF_EUNSUPPORTED;
    }
}

template <bool UP>
int32_t launch_wgrad(const WgradParams& w, int nslab, hipStream_t st) {
    return w.ntn * 256 == w.d ? launch_wgrad_m<UP, 2>(w, nslab, st) : launch_wgrad_m<UP, 1>(w, nslab, st);
}

}  // namespace

extern "C" {

int32_t unif_moe_layer_backward_workspace_size(const unif_moe_config* cfg, size_t* bytes) {
    if (bytes == nullptr) return UNIF_EINVAL;
    const int32_t s = check_backward_shape(cfg);
    if (s != UNIF_OK) return s;
    const unif_moe_config cw = worst_case(*cfg);
    *bytes = plan_backward(dims_of(&cw)).total;
    return UNIF_OK;
}

int32_t unif_moe_layer_backward(const unif_moe_config* cfg_in, const void* X, const uint8_t* valid,
                                const float* W_router, const float* prototypes, const void* W_up,
                                const void* W_down, const void* dY, float* dX, float* dW_up, float* dW_down,
                                float* dW_router, void* workspace, size_t workspace_bytes, void* stream) {
    int32_t s = check_backward_shape(cfg_in);
    if (s != UNIF_OK) return s;
    const unif_moe_config cfg_worst = worst_case(*cfg_in);   // the backward sizes for the worst case
    const unif_moe_config* cfg = &cfg_worst;
    if (cfg->n_tokens > 0 && (X == nullptr || W_router == nullptr || prototypes == nullptr || W_up == nullptr ||
                              W_down == nullptr || dY == nullptr || dX == nullptr))
        return UNIF_EINVAL;
    if (dW_up == nullptr || dW_down == nullptr || dW_router == nullptr) return UNIF_EINVAL;
    const Dims m = dims_of(cfg);
    const BwdPlan bp = plan_backward(m);
    if (workspace == nullptr || workspace_bytes < bp.total) return UNIF_EWORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int cus = cu_count();
    BwdParams p;
    p.N = m.N;
    p.d = m.d;
    p.K = m.K;
    p.B = m.B;
    p.M = m.M;
    p.H = m.H;
    p.alpha_adaptive = cfg->alpha_mode == UNIF_ALPHA_ADAPTIVE;
    p.tau = m.tau;
    p.one_minus_2tau = m.one_minus_2tau;
    p.X = X;
    p.dY = dY;
    p.Wup = W_up;
    p.Wdown = W_down;
    p.Wr = W_router;
    p.dX = dX;
    p.dWup = dW_up;
    p.dWdown = dW_down;
    p.dWr = dW_router;
    // 1. routing and the permutation's tables into the front of the workspace
    char* ws = align_base(workspace);
    const FwdPlan fp = plan_forward(m);
    if (m.N > 0) {
        s = forward_impl(cfg, nullptr, X, valid, W_router, prototypes, W_up, W_down, nullptr, nullptr, ws,
                         bp.fwd, nullptr, stream, true);
        if (s != UNIF_OK) return s;
    }
    p.alpha = reinterpret_cast<const float*>(ws + fp.alpha);
    p.nres = reinterpret_cast<const int*>(ws + fp.nres);
    p.eids = reinterpret_cast<const int*>(ws + fp.eids);
    p.wts = reinterpret_cast<const float*>(ws + fp.wts);
    p.pair_token = reinterpret_cast<const int*>(ws + fp.pair_token);
    p.pair_expert = reinterpret_cast<const int*>(ws + fp.pair_expert);
    p.pair_mask = reinterpret_cast<const uint64_t*>(ws + fp.pair_mask);
    p.pair_of = reinterpret_cast<const int*>(ws + fp.pair_of);
    p.seg_off = reinterpret_cast<const int*>(ws + fp.seg_off);
    p.totals = reinterpret_cast<const int*>(ws + fp.totals);
    p.act = reinterpret_cast<float*>(ws + bp.act);
    p.da = reinterpret_cast<float*>(ws + bp.da);
    p.dcoef = reinterpret_cast<float*>(ws + bp.dcoef);
    p.pw = reinterpret_cast<float*>(ws + bp.pw);
    p.rpart = reinterpret_cast<float*>(ws + bp.rpart);
    p.dxp = reinterpret_cast<float*>(ws + fp.part);
    p.dz = reinterpret_cast<float*>(ws + bp.dz);
    if (m.N == 0) {
        // No tokens: the forward built no tables; the weight gradients are zero.
        const size_t nw[3] = {(size_t)m.K1 * m.H * m.d, (size_t)m.K1 * m.d * m.H, (size_t)m.K1 * m.d};
        float* const outs[3] = {dW_up, dW_down, dW_router};
        for (int i = 0; i < 3; ++i) {
            const unsigned g = (unsigned)std::min<size_t>((nw[i] + 255) / 256, (size_t)cus * 16);
            fill_zero_kernel<<<g, 256, 0, st>>>(reinterpret_cast<uint32_t*>(outs[i]), nw[i]);
            UNIF_LAUNCH_CHECK();
        }
        return UNIF_OK;
    }
    bwd_weight_kernel<<<(unsigned)cus * 4, 256, 0, st>>>(p);
    UNIF_LAUNCH_CHECK();
    const size_t pmax = (size_t)m.N * m.K1;
    u16* const abuf = reinterpret_cast<u16*>(ws + fp.hbuf);
    u16* const gbuf = reinterpret_cast<u16*>(ws + bp.gbuf);
    if (m.bf16) {
        // 2. V^T [K+1, H, d] (rows of dy V as the up kernel's weights) and
        //    K^T [K+1, d, H] (dx_pair = da K as the down kernel's weights)
        int* queues = reinterpret_cast<int*>(ws + bp.queues);
        fill_zero_kernel<<<1, 64, 0, st>>>(reinterpret_cast<uint32_t*>(queues), 32);
        UNIF_LAUNCH_CHECK();
        u16* const wdnT = reinterpret_cast<u16*>(ws + bp.wdnT);
        u16* const wupT = reinterpret_cast<u16*>(ws + fp.wdown16);
        const int nt = m.K1 * (m.d / 64) * (m.H / 64);
        transpose16_kernel<<<(unsigned)ceil_div(nt, 4), 256, 0, st>>>(static_cast<const u16*>(W_down), wdnT, m.d,
                                                                       m.H, nt);
        transpose16_kernel<<<(unsigned)ceil_div(nt, 4), 256, 0, st>>>(static_cast<const u16*>(W_up), wupT, m.H,
                                                                       m.d, nt);
        UNIF_LAUNCH_CHECK();
        // 3. a = x K^T over the slabs (kept in fp16); then dy V: the dy . E
        //    partials, da and w GELU(a)
        UpParams up;
        up.d = m.d;
        up.M = m.M;
        up.B = m.B;
        up.H = m.H;
        up.X = static_cast<const u16*>(X);
        up.Wup = static_cast<const u16*>(W_up);
        up.Hbuf = abuf;
        up.Hsink = abuf + pmax * m.H;
        up.slab_rows = reinterpret_cast<const int*>(ws + fp.slab_rows);
        up.slab_tok = reinterpret_cast<const int*>(ws + fp.slab_tok);
        up.tile_info = reinterpret_cast<const int*>(ws + fp.up_tile_info);
        up.tile_rows = reinterpret_cast<const int*>(ws + fp.up_tile_rows);
        up.totals = p.totals;
        up.queue = queues;
        up.b_up = nullptr;
        up.Gbuf = gbuf;
        up.pw = p.pw;
        float* const dcp = reinterpret_cast<float*>(ws + bp.dcp);
        up.dcp = dcp;
        up.sink_row = (int)pmax;
        const size_t up_lds = (size_t)up_lds_bytes(m.M, up_tm(m.M, m.d));
        const int grid = (cus / kXcds) * kXcds;
        s = launch_up<kEpiPre>(m, grid, up_lds, st, up);
        if (s != UNIF_OK) return s;
        up.X = static_cast<const u16*>(dY);
        up.Wup = wdnT;
        up.queue = queues + 8;
        s = launch_up<kEpiDa>(m, grid, up_lds, st, up);
        if (s != UNIF_OK) return s;
        bwd_dcoef_sum_kernel<<<(unsigned)cus * 4, 256, 0, st>>>(p, dcp);
        UNIF_LAUNCH_CHECK();
        // 4. dx_pair = da K over each pair's blocks
        const DownShape dsh = down_shape(m.d);
        DownParams dn;
        dn.d = m.d;
        dn.M = m.M;
        dn.B = m.B;
        dn.H = m.H;
        dn.ncol = m.d / dsh.bn;
        dn.Hbuf = gbuf;
        dn.zero16 = reinterpret_cast<const u16*>(ws + fp.zero_page);
        dn.Wdown = wupT;
        dn.part = p.dxp;
        dn.part_sink = p.dxp + pmax * m.d;
        dn.rt_info = reinterpret_cast<const int4*>(ws + fp.rt_info);
        dn.rt_masks = reinterpret_cast<const uint64_t*>(ws + fp.rt_masks);
        dn.pair_mask = p.pair_mask;
        dn.slices = reinterpret_cast<const int*>(ws + fp.down_slices);
        dn.queue = queues + 16;
        dn.nsplit = 1;
        dn.split_stride = 0;
        if (dsh.bn == 384)
            s = launch_persistent(down_kernel<2, 3, false>, grid, (size_t)down_lds_bytes(128, 384), st, dn);
        else if (dsh.bn == 256)
            s = launch_persistent(down_kernel<4, 4, false>, grid, (size_t)down_lds_bytes(256, 256), st, dn);
        else
            s = launch_persistent(down_kernel<4, 2, false>, grid, (size_t)down_lds_bytes(256, 128), st, dn);
        if (s != UNIF_OK) return s;
    } else {
        // 2. per pair: tiled fp32 GEMMs over each expert's segment
        const int tiles_h = ceil_div(m.H, kBT), tiles_d = ceil_div(m.d, kBT);
        const unsigned ptiles = (unsigned)ceil_div(m.N, kBT);
        const dim3 g_ch((unsigned)tiles_h, ptiles, (unsigned)m.K1), g_out((unsigned)tiles_d, ptiles, (unsigned)m.K1);
        const unsigned gp = (unsigned)ceil_div(m.N * m.K1, 4);
        bwd_seg_kernel<0><<<g_ch, 256, 0, st>>>(p);
        bwd_seg_kernel<1><<<g_out, 256, 0, st>>>(p);
        bwd_dcoef_kernel<<<gp, 256, 0, st>>>(p);
        bwd_seg_kernel<2><<<g_ch, 256, 0, st>>>(p);
        bwd_seg_kernel<3><<<g_out, 256, 0, st>>>(p);
        UNIF_LAUNCH_CHECK();
    }
    // 5. per token: dX and the router-logit gradients; the router's weight gradient
    bwd_token_kernel<<<(unsigned)ceil_div(m.N, kTokTile), 256, 0, st>>>(p);
    UNIF_LAUNCH_CHECK();
    const dim3 rgrid((unsigned)ceil_div(m.d, kRouterCols), (unsigned)ceil_div(m.K1, 32), kRouterChunks);
    if (m.bf16) bwd_router_kernel<true><<<rgrid, 64, 0, st>>>(p);
    else bwd_router_kernel<false><<<rgrid, 64, 0, st>>>(p);
    UNIF_LAUNCH_CHECK();
    bwd_router_sum_kernel<<<(unsigned)ceil_div(m.K1 * m.d, 256), 256, 0, st>>>(p);
    UNIF_LAUNCH_CHECK();
    // 6. expert weight gradients
    if (m.bf16) {
        WgradParams w;
        w.d = m.d;
        w.M = m.M;
        w.B = m.B;
        w.H = m.H;
        w.ntn = (m.d % 256 == 0) ? m.d / 256 : m.d / 128;
        w.slab_rows = reinterpret_cast<const int*>(ws + fp.slab_rows);
        w.slab_tok = reinterpret_cast<const int*>(ws + fp.slab_tok);
        w.slab_off = reinterpret_cast<const int*>(ws + fp.slab_off);
        w.slab_count = reinterpret_cast<const int*>(ws + fp.slab_count);
        w.Psrc = static_cast<const u16*>(X);
        w.Qsrc = gbuf;
        w.out = dW_up;
        s = launch_wgrad<true>(w, m.nslab, st);
        if (s != UNIF_OK) return s;
        w.Psrc = abuf;
        w.Qsrc = static_cast<const u16*>(dY);
        w.out = dW_down;
        s = launch_wgrad<false>(w, m.nslab, st);
        if (s != UNIF_OK) return s;
    } else {
        const int tiles_h = ceil_div(m.H, kBT), tiles_d = ceil_div(m.d, kBT);
        const dim3 wg_grid((unsigned)(tiles_h * tiles_d), 2, (unsigned)m.K1);
        bwd_wgrad_kernel<<<wg_grid, 256, 0, st>>>(p, tiles_h, tiles_d);
        UNIF_LAUNCH_CHECK();
    }
    return UNIF_OK;
}

int32_t unif_moe_diversity_loss_workspace_size(const unif_moe_config* cfg, size_t* bytes) {
    if (bytes == nullptr) return UNIF_EINVAL;
    const int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    const size_t k1 = (size_t)cfg->n_experts + 1;
    *bytes = 8 * (k1 * k1 + 1) + 256;
    return UNIF_OK;
}

int32_t unif_moe_diversity_loss(const unif_moe_config* cfg, const float* W_router, float lambda, float* loss,
                                float* dW_router, void* workspace, size_t workspace_bytes, void* stream) {
    const int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    if (W_router == nullptr || loss == nullptr || dW_router == nullptr || !std::isfinite(lambda))
        return UNIF_EINVAL;
    size_t need = 0;
    unif_moe_diversity_loss_workspace_size(cfg, &need);
    if (workspace == nullptr || workspace_bytes < need) return UNIF_EWORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    DivParams dp;
    dp.K1 = cfg->n_experts + 1;
    dp.d = cfg->d_model;
    dp.W = W_router;
    char* ws = align_base(workspace);
    dp.G = reinterpret_cast<double*>(ws);
    dp.Ls = dp.G + (size_t)dp.K1 * dp.K1;
    dp.loss = loss;
    dp.dW = dW_router;
    dp.lambda = lambda;
    const int npair = dp.K1 * (dp.K1 + 1) / 2;
    div_gram_kernel<<<(unsigned)ceil_div(npair, 4), 256, 0, st>>>(dp);
    UNIF_LAUNCH_CHECK();
    div_loss_kernel<<<1, 256, 0, st>>>(dp);
    UNIF_LAUNCH_CHECK();
    div_grad_kernel<<<(unsigned)ceil_div(dp.K1 * dp.d, 256), 256, 0, st>>>(dp);
    UNIF_LAUNCH_CHECK();
    return UNIF_OK;
}

int32_t unif_moe_stats_workspace_size(const unif_moe_config* cfg, size_t* bytes) {
    if (bytes == nullptr) return UNIF_EINVAL;
    const int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    *bytes = (size_t)kStWords * 8 + 256;
    return UNIF_OK;
}

int32_t unif_moe_stats(const unif_moe_config* cfg, const unif_moe_routing* routing, const uint8_t* valid,
                       unif_moe_stats_t* host_out, void* workspace, size_t workspace_bytes, void* stream) {
    const int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    if (host_out == nullptr || !record_complete(routing)) return UNIF_EINVAL;
    size_t need = 0;
    unif_moe_stats_workspace_size(cfg, &need);
    if (workspace == nullptr || workspace_bytes < need) return UNIF_EWORKSPACE;
    const Dims m = dims_of(cfg);
    hipStream_t st = static_cast<hipStream_t>(stream);
    unsigned long long* cnt = reinterpret_cast<unsigned long long*>(align_base(workspace));
    fill_zero_kernel<<<1, 256, 0, st>>>(reinterpret_cast<uint32_t*>(cnt), (size_t)kStWords * 2);
    UNIF_LAUNCH_CHECK();
    if (m.N > 0) {
        StatsParams sp;
        sp.N = m.N;
        sp.K = m.K;
        sp.B = m.B;
        sp.valid = valid;
        sp.nsh = routing->n_shared;
        sp.nres = routing->n_res;
        sp.eids = routing->expert_ids;
        sp.out = cnt;
        const int grid = ceil_div(m.N, 256) < 1024 ? ceil_div(m.N, 256) : 1024;
        stats_kernel<<<grid, 256, 0, st>>>(sp);
        UNIF_LAUNCH_CHECK();
    }
    unsigned long long h[kStWords];
    if (hipMemcpyAsync(h, cnt, sizeof(h), hipMemcpyDeviceToHost, st) != hipSuccess) return UNIF_EDEVICE;
    if (hipStreamSynchronize(st) != hipSuccess) return UNIF_EDEVICE;
    std::memset(host_out, 0, sizeof(*host_out));
    host_out->n_valid = (int64_t)h[kStN];
    for (int i = 0; i < 65; ++i) {
        host_out->hist_b[i] = (int64_t)h[kStHistB + i];
        host_out->hist_k[i] = (int64_t)h[kStHistK + i];
        host_out->expert_tokens[i] = (int64_t)h[kStExp + i];
    }
    host_out->activated_blocks = (int64_t)h[kStSumCB];
    const double nv = (double)h[kStN];
    host_out->mean_b = nv > 0 ? (double)h[kStSumB] / nv : 0.0;
    host_out->mean_k = nv > 0 ? (double)h[kStSumK] / nv : 0.0;
    host_out->mean_cb = nv > 0 ? (double)h[kStSumCB] / nv : 0.0;
    host_out->activated_gemm_flops = 4.0 * m.d * m.M * (double)h[kStSumCB];
    host_out->routing_flops = 2.0 * m.d * (1.0 + m.K + m.B) * nv;
    return UNIF_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The layer forward without a caller workspace (unif_moe_layer_forward_static):
// its scratch memory is this file-scope device array, one copy per GPU the
// library's code is loaded on, held until the process ends.
namespace {

constexpr size_t kStaticScratchBytes = UNIF_MOE_STATIC_WORKSPACE_BYTES;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

// Device address of `scratch` on each GPU, looked up once per device with that
// device current (the array's name is a host-side stand-in in host code and
// must never be passed to a kernel or a copy).
constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mutex;

int32_t static_scratch(void** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return UNIF_EDEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return UNIF_EDEVICE;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return UNIF_OK;
}

}  // namespace

extern "C" {

int32_t unif_moe_layer_forward_static(const unif_moe_config* cfg, const void* X, const uint8_t* valid,
                                      const float* W_router, const float* prototypes, const void* W_up,
                                      const void* W_down, void* Y, const unif_moe_routing* routing_out,
                                      void* stream) {
    size_t need = 0;
    const int32_t s = unif_moe_layer_forward_workspace_size(cfg, &need);
    if (s != UNIF_OK) return s;
    if (need > kStaticScratchBytes) return UNIF_EWORKSPACE;
    void* ws = nullptr;
    const int32_t e = static_scratch(&ws);
    if (e != UNIF_OK) return e;
    return forward_impl(cfg, nullptr, X, valid, W_router, prototypes, W_up, W_down, Y, routing_out, ws,
                        kStaticScratchBytes, nullptr, stream);
}

}  // extern "C"

extern "C" {

int32_t unif_moe_forward_status(const unif_moe_config* cfg, const void* workspace, size_t workspace_bytes,
                                int64_t* pairs_needed, void* stream) {
    int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    s = check_forward_shape(cfg);
    if (s != UNIF_OK) return s;
    size_t need = 0;
    unif_moe_layer_forward_workspace_size(cfg, &need);
    if (workspace == nullptr || workspace_bytes < need) return UNIF_EWORKSPACE;
    if (pairs_needed != nullptr) *pairs_needed = 0;
    const Dims m = dims_of(cfg);
    if (m.N == 0) return UNIF_OK;
    // The totals sit at the same offset in the layer's and the block's plans.
    const FwdPlan plan = plan_forward(m);
    const char* ws = align_base(const_cast<void*>(workspace));
    hipStream_t st = static_cast<hipStream_t>(stream);
    int32_t t[8];
    if (hipMemcpyAsync(t, ws + plan.totals, sizeof(t), hipMemcpyDeviceToHost, st) != hipSuccess) return UNIF_EDEVICE;
    if (hipStreamSynchronize(st) != hipSuccess) return UNIF_EDEVICE;
    if (pairs_needed != nullptr) *pairs_needed = t[0];
    return t[5] != 0 ? UNIF_ECAPACITY : UNIF_OK;
}

int32_t unif_moe_forward_work(const unif_moe_config* cfg, const void* workspace, size_t workspace_bytes,
                              unif_moe_work_t* host_out, void* stream) {
    int32_t s = check_config(cfg);
    if (s != UNIF_OK) return s;
    s = check_forward_shape(cfg);
    if (s != UNIF_OK) return s;
    if (host_out == nullptr) return UNIF_EINVAL;
    if (cfg->dtype != UNIF_BF16) return UNIF_EUNSUPPORTED;
    size_t need = 0;
    unif_moe_layer_forward_workspace_size(cfg, &need);
    if (workspace == nullptr || workspace_bytes < need) return UNIF_EWORKSPACE;
    std::memset(host_out, 0, sizeof(*host_out));
    const Dims m = dims_of(cfg);
    if (m.N == 0) return UNIF_OK;
    const FwdPlan plan = plan_forward(m);
    char* ws = align_base(const_cast<void*>(workspace));
    hipStream_t st = static_cast<hipStream_t>(stream);
    unsigned long long* cnt = reinterpret_cast<unsigned long long*>(ws + plan.work);
    const int* totals = reinterpret_cast<const int*>(ws + plan.totals);
    fill_zero_kernel<<<1, 64, 0, st>>>(reinterpret_cast<uint32_t*>(cnt), 2);
    UNIF_LAUNCH_CHECK();
    const DownShape dsh = down_shape(m.d);
    work_kernel<<<(unsigned)std::min<size_t>(ceil_div_sz(plan.max_row_tiles, 256), 1024), 256, 0, st>>>(
        reinterpret_cast<const uint64_t*>(ws + plan.rt_masks), totals, dsh.tm / 32, cnt);
    UNIF_LAUNCH_CHECK();
    int32_t t[8], sl[kXcds + 1];
    unsigned long long g = 0;
    if (hipMemcpyAsync(t, totals, sizeof(t), hipMemcpyDeviceToHost, st) != hipSuccess) return UNIF_EDEVICE;
    if (hipMemcpyAsync(&g, cnt, sizeof(g), hipMemcpyDeviceToHost, st) != hipSuccess) return UNIF_EDEVICE;
    if (hipMemcpyAsync(sl, ws + plan.down_slices, sizeof(sl), hipMemcpyDeviceToHost, st) != hipSuccess)
        return UNIF_EDEVICE;
    if (hipStreamSynchronize(st) != hipSuccess) return UNIF_EDEVICE;
    const double dM = (double)m.M, dd = (double)m.d;
    host_out->pairs = t[0];
    host_out->up_tiles = t[1];
    host_out->down_tiles = t[2];
    host_out->up_mfma_flops = (double)t[1] * up_tm(m.M, m.d) * dM * dd * 2.0;
    host_out->down_mfma_flops = (double)g * 32.0 * dM * dd * 2.0;
    host_out->down_parts = down_splits(m);
    for (int x = 0; x < kXcds; ++x) host_out->down_queued += std::max(0, sl[x + 1] - sl[x]);
    return UNIF_OK;
}

}  // extern "C"

