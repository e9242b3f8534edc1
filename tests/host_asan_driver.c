/* Drives every host-side path of the library that makes no HIP call - the
 * configuration checks, the workspace-size queries and the argument
 * rejections of every entry point - over a grid of valid and invalid
 * configurations. Built together with the library's host code under
 * AddressSanitizer by tests/test_host_asan.py; prints one line per checked
 * expectation that fails and "host paths ok <calls>" at the end. Pointer
 * arguments below are placeholders that every rejected call returns on
 * before touching them. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "unif_moe.h"

static long calls = 0, bad = 0;

static void expect(int32_t got, int32_t want, const char* what, int line) {
    ++calls;
    if (got != want) {
        ++bad;
        printf("line %d: %s returned %d, expected %d\n", line, what, (int)got, (int)want);
    }
}
#define EXPECT(call, want) expect((call), (want), #call, __LINE__)

static unif_moe_config base(void) {
    unif_moe_config c;
    memset(&c, 0, sizeof c);
    c.n_tokens = 50432;
    c.d_model = 768;
    c.n_experts = 16;
    c.n_blocks = 16;
    c.block_width = 192;
    c.dtype = UNIF_BF16;
    c.tau = NAN;
    c.mass_threshold = 0.6f;
    c.max_shared = 16;
    c.alpha_mode = UNIF_ALPHA_ADAPTIVE;
    c.mass_mode = UNIF_MASS_COUPLED;
    c.fixed_k = 1;
    c.select_mode = UNIF_SELECT_PROTOTYPE;
    return c;
}

/* Every size query on cfg; returns the first status (they agree for the
 * shared checks). */
static int32_t sizes(const unif_moe_config* c) {
    size_t n = 0;
    unif_moe_block blk;
    memset(&blk, 0, sizeof blk);
    blk.norm = UNIF_NORM_NONE;
    const int32_t s = unif_moe_route_workspace_size(c, &n);
    unif_moe_layer_forward_workspace_size(c, &n);
    unif_moe_block_forward_workspace_size(c, &blk, &n);
    blk.norm = UNIF_NORM_PRE;
    blk.ln_eps = 1e-6f;
    unif_moe_block_forward_workspace_size(c, &blk, &n);
    blk.norm = UNIF_NORM_POST;
    unif_moe_block_forward_workspace_size(c, &blk, &n);
    unif_moe_layer_backward_workspace_size(c, &n);
    unif_moe_diversity_loss_workspace_size(c, &n);
    unif_moe_stats_workspace_size(c, &n);
    calls += 8;
    return s;
}

int main(void) {
    void* p = (void*)(uintptr_t)4096;
    float* fp = (float*)p;
    size_t n = 0;
    unif_moe_config c = base();

    /* valid layers of several shapes: every query succeeds */
    const int shapes[][6] = {{50432, 768, 16, 16, 192, UNIF_BF16}, {12608, 384, 8, 8, 192, UNIF_BF16},
                             {4096, 1024, 16, 16, 256, UNIF_BF16}, {131072, 1024, 32, 32, 128, UNIF_BF16},
                             {1, 128, 64, 64, 64, UNIF_BF16},       {0, 256, 4, 4, 64, UNIF_BF16},
                             {333, 96, 5, 3, 40, UNIF_F32},         {200, 64, 4, 4, 24, UNIF_F32}};
    for (size_t i = 0; i < sizeof shapes / sizeof shapes[0]; ++i) {
        c = base();
        c.n_tokens = shapes[i][0];
        c.d_model = shapes[i][1];
        c.n_experts = shapes[i][2];
        c.n_blocks = shapes[i][3];
        c.block_width = shapes[i][4];
        c.dtype = shapes[i][5];
        c.max_shared = c.n_blocks;
        EXPECT(sizes(&c), UNIF_OK);
        EXPECT(unif_moe_layer_forward_workspace_size(&c, &n), UNIF_OK);
        EXPECT(unif_moe_layer_backward_workspace_size(&c, &n), UNIF_OK);
    }

    /* one broken field at a time */
    for (int f = 0; f < 20; ++f) {
        c = base();
        int32_t want = UNIF_EINVAL;
        switch (f) {
            case 0: c.n_tokens = -1; break;
            case 1: c.d_model = 0; break;
            case 2: c.n_experts = 0; break;
            case 3: c.n_blocks = 0; break;
            case 4: c.block_width = 0; break;
            case 5: c.dtype = 7; break;
            case 6: c.alpha_mode = 9; break;
            case 7: c.mass_mode = 9; break;
            case 8: c.select_mode = 9; break;
            case 9: c.mass_threshold = 0.0f; break;
            case 10: c.mass_threshold = 1.5f; break;
            case 11: c.max_shared = 17; break;
            case 12: c.n_blocks = 1; c.max_shared = 1; break;
            case 13: c.alpha_mode = UNIF_ALPHA_FIXED; c.alpha_fixed = 1.5f; break;
            case 14: c.mass_mode = UNIF_MASS_TOPK; c.fixed_k = 17; break;
            case 15: c.tau = 0.5f; break;
            case 16: c.n_experts = 65; want = UNIF_EUNSUPPORTED; break;
            case 17: c.n_blocks = 65; c.max_shared = 65; want = UNIF_EUNSUPPORTED; break;
            case 18: c.n_tokens = 0x7fffffff; want = UNIF_EUNSUPPORTED; break;
            case 19: c.mass_threshold = NAN; break;
        }
        EXPECT(sizes(&c), want);
        EXPECT(unif_moe_route(&c, p, NULL, fp, fp, NULL, p, (size_t)1 << 40, NULL), want);
    }
    /* bf16 shapes the GEMM engines do not take */
    c = base();
    c.d_model = 800;
    EXPECT(unif_moe_layer_forward_workspace_size(&c, &n), UNIF_EUNSUPPORTED);
    c = base();
    c.block_width = 96;
    EXPECT(unif_moe_layer_forward_workspace_size(&c, &n), UNIF_EUNSUPPORTED);
    c = base();
    c.block_width = 320;
    EXPECT(unif_moe_layer_forward_workspace_size(&c, &n), UNIF_EUNSUPPORTED);

    /* NULL outputs and small workspaces, for every entry point */
    c = base();
    unif_moe_routing rec = {fp, (int32_t*)p, (uint64_t*)p, (int32_t*)p, (int32_t*)p, fp};
    unif_moe_routing half = rec;
    half.weights = NULL;
    EXPECT(unif_moe_route_workspace_size(&c, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_route_workspace_size(NULL, &n), UNIF_EINVAL);
    EXPECT(unif_moe_route(&c, p, NULL, fp, fp, NULL, p, (size_t)1 << 40, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_route(&c, p, NULL, fp, fp, &half, p, (size_t)1 << 40, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_route(&c, p, NULL, fp, fp, &rec, p, 1, NULL), UNIF_EWORKSPACE);
    EXPECT(unif_moe_layer_forward(&c, p, NULL, fp, fp, p, p, NULL, NULL, p, (size_t)1 << 40, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_layer_forward(&c, p, NULL, fp, fp, p, p, p, &half, p, (size_t)1 << 40, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_layer_forward(&c, p, NULL, fp, fp, p, p, p, NULL, p, 16, NULL), UNIF_EWORKSPACE);
    EXPECT(unif_moe_layer_forward(&c, p, NULL, fp, fp, p, p, p, NULL, NULL, 0, NULL), UNIF_EWORKSPACE);
    void* ev[7] = {p, p, p, p, p, p, NULL};
    EXPECT(unif_moe_layer_forward_profiled(&c, p, NULL, fp, fp, p, p, p, NULL, p, (size_t)1 << 40, ev, 7, NULL),
           UNIF_EINVAL);
    EXPECT(unif_moe_layer_forward_profiled(&c, p, NULL, fp, fp, p, p, p, NULL, p, (size_t)1 << 40, ev, 6, NULL),
           UNIF_EINVAL);
    unif_moe_block blk;
    memset(&blk, 0, sizeof blk);
    blk.norm = UNIF_NORM_PRE;
    blk.ln_eps = 1e-6f;
    EXPECT(unif_moe_block_forward(&c, &blk, p, NULL, fp, fp, p, p, p, NULL, p, (size_t)1 << 40, NULL),
           UNIF_EINVAL); /* no gamma / beta */
    EXPECT(unif_moe_block_forward(&c, NULL, p, NULL, fp, fp, p, p, p, NULL, p, (size_t)1 << 40, NULL),
           UNIF_EINVAL);
    blk.norm = 5;
    EXPECT(unif_moe_block_forward_workspace_size(&c, &blk, &n), UNIF_EINVAL);
    blk.norm = UNIF_NORM_PRE;
    blk.ln_eps = -1.0f;
    EXPECT(unif_moe_block_forward_workspace_size(&c, &blk, &n), UNIF_EINVAL);
    blk.ln_eps = INFINITY;
    EXPECT(unif_moe_block_forward_workspace_size(&c, &blk, &n), UNIF_EINVAL);
    EXPECT(unif_moe_layer_backward(&c, p, NULL, fp, fp, p, p, NULL, fp, fp, fp, fp, p, (size_t)1 << 40, NULL),
           UNIF_EINVAL);
    EXPECT(unif_moe_layer_backward(&c, p, NULL, fp, fp, p, p, p, fp, NULL, fp, fp, p, (size_t)1 << 40, NULL),
           UNIF_EINVAL);
    EXPECT(unif_moe_layer_backward(&c, p, NULL, fp, fp, p, p, p, fp, fp, fp, fp, p, 16, NULL), UNIF_EWORKSPACE);
    EXPECT(unif_moe_diversity_loss(&c, NULL, 1.0f, fp, fp, p, 1 << 20, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_diversity_loss(&c, fp, NAN, fp, fp, p, 1 << 20, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_diversity_loss(&c, fp, 1.0f, fp, fp, p, 8, NULL), UNIF_EWORKSPACE);
    unif_moe_stats_t st;
    EXPECT(unif_moe_stats(&c, NULL, NULL, &st, p, 1 << 20, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_stats(&c, &rec, NULL, NULL, p, 1 << 20, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_stats(&c, &rec, NULL, &st, p, 8, NULL), UNIF_EWORKSPACE);
    unif_moe_work_t w;
    EXPECT(unif_moe_forward_work(&c, p, (size_t)1 << 40, NULL, NULL), UNIF_EINVAL);
    EXPECT(unif_moe_forward_work(&c, p, 8, &w, NULL), UNIF_EWORKSPACE);
    c.dtype = UNIF_F32;
    c.d_model = 96;
    c.block_width = 40;
    EXPECT(unif_moe_forward_work(&c, p, (size_t)1 << 40, &w, NULL), UNIF_EUNSUPPORTED);
    /* the static forward: a layer beyond its scratch, and a bad config */
    c = base();
    EXPECT(unif_moe_layer_forward_static(&c, p, NULL, fp, fp, p, p, p, NULL, NULL), UNIF_EWORKSPACE);
    c.n_experts = 0;
    EXPECT(unif_moe_layer_forward_static(&c, p, NULL, fp, fp, p, p, p, NULL, NULL), UNIF_EINVAL);
    /* status strings */
    for (int s = -8; s <= 3; ++s) {
        const char* t = unif_moe_status_string(s);
        ++calls;
        if (t == NULL || strlen(t) == 0) {
            ++bad;
            printf("status %d: empty string\n", s);
        }
    }
    printf("host paths %s %ld\n", bad ? "FAILED" : "ok", calls);
    return bad ? 1 : 0;
}
