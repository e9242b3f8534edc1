/*
 * unif_moe.h - C ABI of the MI355X (gfx950) library for the forward pass of
 * one UniF-MoE feed-forward layer ("Share First, Route What Remains",
 * Sec. III).
 *
 * The layer holds one shared expert E_shr and K residual experts E_1..E_K,
 * all upcycled from one FFN of width H and split into B aligned blocks of
 * M = H / B channels (Sec. III-A). For each token x (a row of X):
 *   alpha = tau + (1 - 2 tau) sigmoid(x W_shr), tau = (B-1)/B^2   (Eq. alpha)
 *   b     = round(B alpha)                                         (Eq. block-count)
 *   I_shr = the b blocks with the largest x mu_c                   (Eq. block-priority,
 *           I_res = the other blocks                                shared-indices,
 *                                                                   residual-indices)
 *   s     = softmax(x W_g) over the K residual experts            (Eq. residual-router-score)
 *   q, p  = experts by decreasing s and their affinities           (Eq. sorted-affinity)
 *   k     = smallest n with p_1 + .. + p_n >= 1 - alpha            (Eq. beta, expert-count)
 *   y     = alpha sum_{c in I_shr} E_shr^(c)(x)
 *           + sum_{i <= k} p_i sum_{c in I_res} E_{q_i}^(c)(x)     (Eq. output)
 * with E_j^(c)(x) = sum_{h in block c} GELU(x K_j[:,h]) V_j[h,:]   (Eq. block-expert-output),
 * GELU in its exact erf form and no biases.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every tensor pointer is a DEVICE pointer owned by the caller. The
 *   library allocates and frees nothing and keeps no state between calls.
 * - Calls are asynchronous on `stream` (a hipStream_t; NULL is the null
 *   stream), except unif_moe_stats, which synchronises it.
 * - Arguments are validated on the host before any HIP call; a rejected
 *   call launches nothing and leaves every buffer untouched.
 * - Scratch memory comes from a caller-provided `workspace` of at least the
 *   size reported by the matching *_workspace_size function (any alignment;
 *   the library aligns its regions to 256 bytes inside it). Calls that share
 *   a workspace must be ordered on one stream.
 * - Row-major layouts. bf16 data is IEEE binary32 with the low 16 bits
 *   dropped (bfloat16), passed as 16-bit words; conversions to bf16 round
 *   to nearest even. The router and the block prototypes are always fp32.
 * - Inputs must be finite (documented, not checked).
 * - Padded tokens (valid[t] == 0) are skipped: their routing record is
 *   alpha = 0, b = k = 0, mask = 0, expert ids -1, weights 0, their output
 *   row is zero, and they count nowhere in the statistics.
 */
#ifndef UNIF_MOE_H
#define UNIF_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes (every entry point returns one as int32_t). */
#define UNIF_OK            0   /* success                                        */
#define UNIF_EINVAL       (-1) /* invalid argument: NULL pointer, bad size/mode  */
#define UNIF_EWORKSPACE   (-2) /* workspace smaller than the reported size       */
#define UNIF_EDEVICE      (-3) /* a HIP launch or runtime call failed            */
#define UNIF_EUNSUPPORTED (-4) /* valid layer the library does not implement   */
#define UNIF_ECAPACITY    (-5) /* the routing needs more (token, expert) pairs
                                  than cfg->max_pairs (unif_moe_forward_status) */

/* Element type of X, W_up, W_down and Y. */
#define UNIF_F32  0
#define UNIF_BF16 1

/* alpha_mode: ADAPTIVE is Eq. alpha; FIXED uses alpha_fixed for every token
 * (the fixed-alpha ablation, Table mechanism-ablation). */
#define UNIF_ALPHA_ADAPTIVE 0
#define UNIF_ALPHA_FIXED    1

/* mass_mode: the target that the prefix sums P_n of Eq. expert-count must
 * reach. COUPLED: min(1 - alpha, mass_threshold); with mass_threshold = 1
 * this is Eq. beta / expert-count exactly. FIXED: mass_threshold for every
 * token. TOPK: k = fixed_k (the top-k residual-activation ablation). */
#define UNIF_MASS_COUPLED 0
#define UNIF_MASS_FIXED   1
#define UNIF_MASS_TOPK    2

/* select_mode: PROTOTYPE is Eq. shared-indices (the b blocks of largest
 * x mu_c, ties to the lower block index); PREFIX takes blocks 0..b-1 (the
 * prefix-selection ablation). */
#define UNIF_SELECT_PROTOTYPE 0
#define UNIF_SELECT_PREFIX    1

/* Layer description (Sec. III). */
typedef struct unif_moe_config {
    int32_t n_tokens;       /* N >= 0, rows of X                                   */
    int32_t d_model;        /* d > 0                                               */
    int32_t n_experts;      /* K in [1, 64] residual experts; the shared expert is
                               stored in addition, as expert 0                     */
    int32_t n_blocks;       /* B in [1, 64] (>= 2 in ADAPTIVE mode, Sec. III-B)    */
    int32_t block_width;    /* M = H / B channels per block                        */
    int32_t dtype;          /* UNIF_F32 or UNIF_BF16                               */
    float   tau;            /* tau of Eq. alpha; NaN selects (B-1)/B^2. Must lie
                               in [0, 1/2). 1 - 2 tau is evaluated in fp32.        */
    float   mass_threshold; /* t in (0, 1], see mass_mode                          */
    int32_t max_shared;     /* cap on b applied after Eq. block-count, in [0, B]   */
    int32_t alpha_mode;     /* UNIF_ALPHA_*                                        */
    float   alpha_fixed;    /* alpha in [0, 1] when alpha_mode == FIXED            */
    int32_t mass_mode;      /* UNIF_MASS_*                                         */
    int32_t fixed_k;        /* k in [1, K] when mass_mode == TOPK                  */
    int32_t select_mode;    /* UNIF_SELECT_*                                       */
    int32_t max_pairs;      /* >= 0: capacity of the forward's workspace in (token,
                               expert) pairs, sum over valid tokens of 1 + k; 0 (or
                               at least N (K+1)) sizes it for the worst case
                               N (K+1). Read by the forward entry points only (see
                               unif_moe_layer_forward); the backward always sizes
                               for the worst case.                                 */
} unif_moe_config;

/* Per-token routing record, device arrays written by the library. Residual
 * experts are numbered 1..K as E_1..E_K in the paper; index 0 of the expert
 * weights is the shared expert.
 *   alpha[N]          shared demand alpha (Eq. alpha), fp32
 *   n_shared[N]       b, shared block count after clamp and cap (Eq. block-count)
 *   shared_mask[N]    bit c set <=> block c in I_shr (Eq. shared-indices)
 *   n_res[N]          k, residual expert count (Eq. expert-count)
 *   expert_ids[N*K]   q_1..q_K, all K experts by decreasing affinity (ties to
 *                     the lower index) (Eq. sorted-affinity)
 *   weights[N*K]      p_1..p_K, their softmax affinities (fp32)            */
typedef struct unif_moe_routing {
    float*    alpha;
    int32_t*  n_shared;
    uint64_t* shared_mask;
    int32_t*  n_res;
    int32_t*  expert_ids;
    float*    weights;
} unif_moe_routing;

/* Counts over valid tokens (host structure filled by unif_moe_stats). */
typedef struct unif_moe_stats_t {
    int64_t n_valid;
    int64_t hist_b[65];           /* tokens with b = i                             */
    int64_t hist_k[65];           /* tokens with k = i                             */
    int64_t expert_tokens[65];    /* [0]: tokens on the shared expert (all valid);
                                     [j]: tokens routed to residual expert j       */
    int64_t activated_blocks;     /* sum of C_B = b + k (B - b) (Eq. block-compute) */
    double  mean_b, mean_k, mean_cb;
    double  activated_gemm_flops; /* 4 d M sum C_B: up- and down-projection FLOPs  */
    double  routing_flops;        /* 2 d (1 + K + B) per valid token               */
} unif_moe_stats_t;

/* Workspace needed by unif_moe_route for this configuration (bytes, may be
 * 0). Host only; no HIP call. Returns UNIF_OK, UNIF_EINVAL or
 * UNIF_EUNSUPPORTED exactly as unif_moe_route would. */
int32_t unif_moe_route_workspace_size(const unif_moe_config* cfg, size_t* bytes);

/* Routing of Sec. III-B and III-C for every token (no expert evaluation).
 *   X          [N, d] fp32 or bf16 (cfg->dtype)
 *   valid      [N] uint8, nonzero = real token; NULL means all valid
 *   W_router   [K+1, d] fp32: row 0 is W_shr, row j is W_j (the columns of
 *              the augmented router W_g* of Eq. augmented-router)
 *   prototypes [B, d] fp32: row c is the block prototype mu_c
 *              (Eq. block-prototype; weight-only, so precomputed by the caller)
 *   out        record arrays (all six required)
 * Errors: UNIF_EINVAL, UNIF_EWORKSPACE, UNIF_EUNSUPPORTED before any launch;
 * UNIF_EDEVICE if a launch fails. */
int32_t unif_moe_route(const unif_moe_config* cfg, const void* X, const uint8_t* valid,
                       const float* W_router, const float* prototypes,
                       const unif_moe_routing* out, void* workspace, size_t workspace_bytes,
                       void* stream);

/* Workspace needed by unif_moe_layer_forward (bytes). Host only. With
 * cfg->max_pairs = 0 the size covers the worst case (every token routed to
 * all K residual experts), so the forward never reads counts back to the
 * host; a capacity max_pairs > 0 sizes the pair-indexed buffers (the fp16
 * activations, the per-expert rows, the pair and slab lists, the down-tile
 * tables) for that many pairs instead, which shrinks the workspace by about
 * N (K+1) / max_pairs for large layers. */
int32_t unif_moe_layer_forward_workspace_size(const unif_moe_config* cfg, size_t* bytes);

/* Forward pass of the layer: routing, token permutation, block-sparse expert
 * FFNs and the weighted merge of Eq. output.
 *   X, valid, W_router, prototypes   as for unif_moe_route
 *   W_up   [K+1, H, d] (cfg->dtype): expert e's row h is the key K_e[:, h]
 *          (the [out, in] weight of the FFN's first linear layer);
 *          expert 0 is the shared expert
 *   W_down [K+1, d, H] (cfg->dtype): expert e's row j holds V_e[:, j], i.e.
 *          V_e stored column-major (the [out, in] weight of the second
 *          linear layer)
 *   Y      [N, d] (cfg->dtype), written for every row (zero for padded rows)
 *   routing_out  optional record (NULL: kept inside the workspace)
 * Precision of the bf16 path: the up-projection multiplies bf16 values
 * (exact products, fp32 accumulation); the GELU activations are rounded to
 * fp16 and multiplied with an fp16 copy of W_down (made in the workspace at
 * each call; exact for bf16 magnitudes in [2^-17, 65504], larger ones become
 * infinities), accumulating in fp32; the per-expert outputs E_j(x) stay fp32
 * and Y is rounded once to bf16. Activations beyond 65504 in magnitude are
 * not representable in fp16 and make the output infinite. The merge sums in
 * a fixed order (shared expert, then q_1..q_k), so repeated calls give
 * bitwise-identical Y.
 * Capacity: when cfg->max_pairs > 0 and the routing of this call needs more
 * (token, expert) pairs than that, the call still writes the routing record
 * but runs no expert FFN and writes Y = 0; the overflow is detected on the
 * device (nothing is read back) and reported afterwards by
 * unif_moe_forward_status. The result never depends on the capacity
 * otherwise.
 * Requires, for bf16: d % 128 == 0, M % 64 == 0, M <= 256; for fp32:
 * H = B M <= 16384. Otherwise UNIF_EUNSUPPORTED. */
int32_t unif_moe_layer_forward(const unif_moe_config* cfg, const void* X, const uint8_t* valid,
                               const float* W_router, const float* prototypes,
                               const void* W_up, const void* W_down, void* Y,
                               const unif_moe_routing* routing_out,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Instrumented unif_moe_layer_forward for measurement: identical work and
 * result, and additionally records the caller's events (hipEvent_t handles,
 * created by the caller, recorded on `stream`) at the phase boundaries:
 *   events[0] before the first launch
 *   events[1] right after events[0] (kept for the layout of the array: the
 *             fp16 copy of W_down runs inside the routing launches)
 *   events[2] after routing (split, route, and the fp16 copy of W_down on
 *             the bf16 path)
 *   events[3] after the permutation (scan, scatter, slab lists)
 *   events[4] after the up-projection
 *   events[5] after the down-projection
 *   events[6] after the weighted merge
 * n_events must be 7. In the fp32 path events[4] and events[5] both follow
 * the per-pair FFN. Errors as unif_moe_layer_forward; UNIF_EINVAL for a NULL
 * event array or n_events != 7. */
int32_t unif_moe_layer_forward_profiled(const unif_moe_config* cfg, const void* X,
                                        const uint8_t* valid, const float* W_router,
                                        const float* prototypes, const void* W_up,
                                        const void* W_down, void* Y,
                                        const unif_moe_routing* routing_out, void* workspace,
                                        size_t workspace_bytes, void* const* events,
                                        int32_t n_events, void* stream);

/* The transformer block around the layer (the paper converts FFN layers of
 * a pre-LN DeiT and a post-LN BERT backbone; its equations leave biases
 * out). With F the layer above plus FFN biases:
 *   UNIF_NORM_NONE  y = [x +] F(x)
 *   UNIF_NORM_PRE   y = [x +] F(LN(x))     (pre-LN block, as in DeiT)
 *   UNIF_NORM_POST  y = LN([x +] F(x))     (post-LN block, as in BERT)
 * where [x +] is the residual add (switched by `residual`) and
 *   LN(v) = (v - mean(v)) / sqrt(var(v) + eps) * gamma + beta
 * with the biased variance over the d features. Biases (readings, since the
 * paper does not define them per block):
 *   b_up (b1) enters every active channel before the GELU:
 *     GELU(x K_j[:, h] + b1_j[h]);
 *   b_down (b2) of expert j is split over its blocks in proportion: a
 *     pathway that runs the set C of blocks adds (|C| / B) b2_j, so the
 *     shared part (alpha-weighted, C = I_shr) and the residual part
 *     (p_i-weighted, C = I_res) of one expert sum to its whole FFN.
 * Padded tokens have F = 0 (no bias terms); the rest of the block applies. */
#define UNIF_NORM_NONE 0
#define UNIF_NORM_PRE  1
#define UNIF_NORM_POST 2

typedef struct unif_moe_block {
    int32_t      norm;      /* UNIF_NORM_*                                         */
    int32_t      residual;  /* nonzero: add the block input x                      */
    float        ln_eps;    /* eps > 0, finite (unused for UNIF_NORM_NONE)         */
    const float* ln_gamma;  /* [d] fp32 device array (required unless NONE)        */
    const float* ln_beta;   /* [d] fp32 device array (required unless NONE)        */
    const float* b_up;      /* [K+1, H] fp32 device array, row e = b1 of expert e;
                               NULL: no up-projection bias. 16-byte aligned for
                               bf16 layers                                         */
    const float* b_down;    /* [K+1, d] fp32 device array, row e = b2 of expert e;
                               NULL: no down-projection bias. 16-byte aligned
                               for bf16 layers                                     */
} unif_moe_block;

/* Workspace needed by unif_moe_block_forward (bytes). Host only. Returns
 * UNIF_OK, UNIF_EINVAL or UNIF_EUNSUPPORTED exactly as the forward would
 * before its pointer checks. */
int32_t unif_moe_block_forward_workspace_size(const unif_moe_config* cfg,
                                              const unif_moe_block* blk, size_t* bytes);

/* Forward pass of the block around the layer (see unif_moe_block): the
 * layer's routing, permutation and block-sparse FFNs run on the FFN input
 * (LN(x) for UNIF_NORM_PRE, else x), with the biases of `blk`; the merge of
 * Eq. output then adds the b2 shares, the residual x and, for
 * UNIF_NORM_POST, the LayerNorm. Arguments as unif_moe_layer_forward, plus
 * `blk` (host structure holding device pointers).
 * Precision: LN statistics and the normalisation run in fp64 and are rounded
 * once to the layer's format (to nearest even; for bf16 through
 * round-to-odd fp32, which equals direct rounding for normal results).
 * Pre-LN: LN(x) is stored in the layer's format, as the FFN's input.
 * Requires what unif_moe_layer_forward requires, and d <= 40960 for
 * UNIF_NORM_POST (one fp32 row in LDS); otherwise UNIF_EUNSUPPORTED.
 * Errors: UNIF_EINVAL (also for a NULL blk, an unknown norm, a bad eps, a
 * missing gamma/beta or a misaligned bias), UNIF_EWORKSPACE,
 * UNIF_EUNSUPPORTED, UNIF_EDEVICE. */
int32_t unif_moe_block_forward(const unif_moe_config* cfg, const unif_moe_block* blk,
                               const void* X, const uint8_t* valid, const float* W_router,
                               const float* prototypes, const void* W_up, const void* W_down,
                               void* Y, const unif_moe_routing* routing_out, void* workspace,
                               size_t workspace_bytes, void* stream);

/* Workspace needed by unif_moe_layer_backward (bytes). Host only. It holds
 * the forward's workspace (routing record, pair tables, the H buffer and
 * the fp32 per-pair rows, which take dx per pair), and, for bf16 layers, a
 * second H-shaped buffer ((N(K+1) + 1) H bf16 values), a transposed copy of
 * W_down and 8 B N(K+1) bytes of per-block partial sums; for fp32 layers
 * 8 H N(K+1) bytes of fp32 intermediates. */
int32_t unif_moe_layer_backward_workspace_size(const unif_moe_config* cfg, size_t* bytes);

/* Backward pass of the layer for a training step: the gradients of
 * sum(dY * Y) with Y the output of unif_moe_layer_forward for the same
 * arguments. Routing and the permutation are recomputed inside (same
 * kernels, so the same discrete decisions). Readings, since the paper gives
 * no gradients: the decisions b, I_shr, the expert order q and k are held
 * fixed (they are piecewise constant); gradients flow through alpha (Eq.
 * alpha) to W_shr and x, through the selected affinities p_i (softmax of
 * Eq. residual-router-score) to W_1..W_K and x, and through the expert FFNs
 * of Eq. block-expert-output; the prototypes get none. Padded tokens get
 * dX = 0 and contribute nothing.
 *   dY         [N, d] (cfg->dtype)
 *   dX         [N, d] fp32, written
 *   dW_up      [K+1, H, d] fp32, written (layout of W_up)
 *   dW_down    [K+1, d, H] fp32, written (layout of W_down)
 *   dW_router  [K+1, d] fp32, written (layout of W_router)
 * Every gradient is bitwise repeatable: each sum runs in a fixed order (the
 * expert weight gradients over each (expert, block)'s rows in token order).
 * bf16 layers run on the matrix cores over the (pair, block) rows the
 * forward runs, never over inactive blocks: a = x K^T kept in fp16; dy V
 * (bf16 products, fp32 sums) gives the pair's d loss / d weight (sum of
 * GELU(a) . dy V over its blocks, fp32), then
 * d loss / da = w (dy V) GELU'(a) and w GELU(a), both rounded to bf16, which
 * feed dx = sum over blocks of (d loss / da) K and the weight gradients
 * (bf16 products, fp32 sums). fp32 layers run on the vector units in fp32
 * (tiled GEMMs over each expert's pairs, dense over H and masked to the
 * pair's blocks) and require N <= 8,388,480. Requires d % 8 == 0 and what
 * unif_moe_layer_forward requires; otherwise UNIF_EUNSUPPORTED. Errors as
 * unif_moe_layer_forward. */
int32_t unif_moe_layer_backward(const unif_moe_config* cfg, const void* X, const uint8_t* valid,
                                const float* W_router, const float* prototypes, const void* W_up,
                                const void* W_down, const void* dY, float* dX, float* dW_up,
                                float* dW_down, float* dW_router, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Workspace needed by unif_moe_diversity_loss (bytes): 8 ((K+1)^2 + 1)
 * bytes plus alignment. Host only. */
int32_t unif_moe_diversity_loss_workspace_size(const unif_moe_config* cfg, size_t* bytes);

/* Gram diversity loss of the augmented router (Eq. diversity-loss, part of
 * the training objective of Eq. loss): with W* the d x (K+1) matrix whose
 * columns are the rows of W_router (W_shr, W_1..W_K),
 *   *loss = L_div = || W*^T W* - I_{K+1} ||_F          (device fp32, written)
 *   dW_router += lambda * dL_div / dW_router             (device fp32 [K+1, d], updated)
 * where dL_div / dW_router = (2 / L_div) (G - I) W_router, G = W_router
 * W_router^T, and nothing is added when L_div = 0 or lambda = 0 (so a
 * training step calls it after unif_moe_layer_backward with the loss
 * weight lambda). Arithmetic in fp64 with fixed summation orders (bitwise
 * repeatable); the outputs are rounded to fp32 once. Only K and d of cfg
 * are read (cfg is validated as for the layer).
 * Errors: UNIF_EINVAL (NULL W_router, loss or dW_router, non-finite
 * lambda), UNIF_EWORKSPACE, UNIF_EDEVICE. */
int32_t unif_moe_diversity_loss(const unif_moe_config* cfg, const float* W_router, float lambda, float* loss,
                                float* dW_router, void* workspace, size_t workspace_bytes, void* stream);

/* Scratch memory of unif_moe_layer_forward_static on each GPU (bytes). */
#define UNIF_MOE_STATIC_WORKSPACE_BYTES ((size_t)128 << 20)

/* unif_moe_layer_forward for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. Same arguments, work and result as unif_moe_layer_forward, but
 * no caller workspace: the scratch memory is a file-scope device array of
 * UNIF_MOE_STATIC_WORKSPACE_BYTES held by each GPU that the library's code is
 * loaded on until the process ends. The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); its first call on a device looks
 * up the array's device address once (hipGetSymbolAddress).
 * All calls on one GPU share that GPU's array and every call clears what it
 * needs zeroed; calls that overlap in time on one GPU (other streams or host
 * threads) race on it and must be ordered by the caller.
 * Errors: as unif_moe_layer_forward; UNIF_EWORKSPACE when the layer needs
 * more scratch than UNIF_MOE_STATIC_WORKSPACE_BYTES (the size reported by
 * unif_moe_layer_forward_workspace_size; checked on the host before any HIP
 * call); UNIF_EDEVICE when the array's address cannot be obtained. */
int32_t unif_moe_layer_forward_static(const unif_moe_config* cfg, const void* X, const uint8_t* valid,
                                      const float* W_router, const float* prototypes, const void* W_up,
                                      const void* W_down, void* Y, const unif_moe_routing* routing_out,
                                      void* stream);

/* Workspace needed by unif_moe_stats (bytes). Host only. */
int32_t unif_moe_stats_workspace_size(const unif_moe_config* cfg, size_t* bytes);

/* Counts of Sec. III-E over a routing record produced by unif_moe_route or
 * unif_moe_layer_forward for the same cfg and valid mask: histograms of b
 * and k, tokens per expert, C_B = b + k (B - b) (Eq. block-compute) and the
 * activated expert-GEMM FLOPs 4 d M C_B. Reduces on the device, copies the
 * counts to *host_out and synchronises `stream`. */
int32_t unif_moe_stats(const unif_moe_config* cfg, const unif_moe_routing* routing,
                       const uint8_t* valid, unif_moe_stats_t* host_out,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Work that a bf16 forward executed (host structure filled by
 * unif_moe_forward_work): the up-projection computes whole tiles of its
 * slabs' rows, the down-projection each 32-row group over the blocks any of
 * its rows uses (the activated work is 4 d M sum C_B, unif_moe_stats). */
typedef struct unif_moe_work_t {
    int64_t pairs;            /* (token, expert) pairs                            */
    int64_t up_tiles;         /* up-projection tiles                              */
    int64_t down_tiles;       /* down-projection tiles (row tiles x column tiles) */
    double  up_mfma_flops;    /* matrix-core FLOPs the up-projection executed     */
    double  down_mfma_flops;  /* matrix-core FLOPs the down-projection executed   */
    int64_t down_parts;       /* parts each down tile's block union is split into */
    int64_t down_queued;      /* down tiles the per-XCD queues hold, summed over  */
                              /* the queues: down_tiles x down_parts when each    */
                              /* tile is queued exactly once                      */
} unif_moe_work_t;

/* Reads the tile tables that the last unif_moe_layer_forward (or
 * _profiled / _static: the latter's workspace is not reachable here) left in
 * `workspace` for this cfg and fills *host_out; synchronises `stream`.
 * bf16 layers only (UNIF_EUNSUPPORTED otherwise). Errors: UNIF_EINVAL,
 * UNIF_EWORKSPACE, UNIF_EUNSUPPORTED, UNIF_EDEVICE. Follows the shape rules
 * of unif_moe_layer_forward. */
int32_t unif_moe_forward_work(const unif_moe_config* cfg, const void* workspace, size_t workspace_bytes,
                              unif_moe_work_t* host_out, void* stream);

/* Outcome of the last forward (unif_moe_layer_forward, _profiled or
 * unif_moe_block_forward) that used `workspace` with this cfg: UNIF_OK, or
 * UNIF_ECAPACITY when its routing needed more pairs than cfg->max_pairs (its
 * Y is then zero). *pairs_needed (host, may be NULL) receives the number of
 * (token, expert) pairs that routing produced. Copies two words to the host
 * and synchronises `stream`. Errors: UNIF_EINVAL, UNIF_EWORKSPACE,
 * UNIF_EUNSUPPORTED, UNIF_EDEVICE, as unif_moe_layer_forward. */
int32_t unif_moe_forward_status(const unif_moe_config* cfg, const void* workspace, size_t workspace_bytes,
                                int64_t* pairs_needed, void* stream);

/* Static text for a status code ("unknown status" for other values). */
const char* unif_moe_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* UNIF_MOE_H */
