/* Host sanitizer driver for the library's argument validation (test
 * infrastructure): every entry point of include/cola.h called with invalid
 * descriptors, NULL and misaligned pointers, short workspaces, overflowing
 * sizes and bad enums, all of which must be refused before anything is
 * enqueued (so no GPU is needed), plus the workspace and saved-size queries
 * over many shapes.  Built with AddressSanitizer and
 * UndefinedBehaviorSanitizer on the host code; any report fails the run. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "cola.h"

#define FAKE ((void*)0x1000)
static int failures = 0;

static void expect(int got, int want, const char* what) {
    if (got != want) {
        printf("FAIL %s: status %d, expected %d\n", what, got, want);
        failures++;
    }
}

int main(void) {
    /* layer descriptors: sizes over a sweep, then refusals */
    for (int64_t T = 0; T < 3000; T += 997)
        for (int64_t r = 1; r < 600; r += 131)
            for (int phase = -1; phase < 5; ++phase) {
                cola_desc d = {T, 300, 517, r, 0, 0, 0, COLA_BF16, COLA_ACT_SILU, (int)(r & 1)};
                (void)cola_workspace_bytes(&d, phase);
                d.dtype = COLA_F32;
                (void)cola_workspace_bytes(&d, phase);
            }
    cola_desc ok = {64, 32, 24, 8, 0, 0, 0, COLA_BF16, COLA_ACT_SILU, 0};
    cola_desc d = ok;
    expect(cola_fwd(NULL, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL), COLA_ERR_INVALID_ARG, "NULL desc");
    d.act = 9;
    expect(cola_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL), COLA_ERR_INVALID_ARG, "bad act");
    d = ok; d.dtype = 7;
    expect(cola_bwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL),
           COLA_ERR_INVALID_ARG, "bad dtype");
    d = ok; d.T = -1;
    expect(cola_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL), COLA_ERR_BAD_SHAPE, "T < 0");
    d = ok; d.ldx = 31;
    expect(cola_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL), COLA_ERR_BAD_SHAPE, "ld < width");
    d = ok; d.T = (int64_t)1 << 62;
    expect(cola_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL), COLA_ERR_BAD_SHAPE, "overflow");
    d = ok; d.recompute = 1;
    expect(cola_fwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL), COLA_ERR_INVALID_ARG,
           "H with CoLA-M");
    d = ok;
    expect(cola_bwd(&d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, NULL), COLA_ERR_WORKSPACE,
           "short workspace");
    cola_desc big = {32768, 2048, 2048, 512, 0, 0, 0, COLA_BF16, COLA_ACT_SILU, 0};
    expect(cola_bwd_scratch(&big, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, NULL), COLA_ERR_SCRATCH,
           "scratch too small");
    expect(cola_infer(NULL, FAKE, FAKE, FAKE, FAKE, FAKE, 0, NULL), COLA_ERR_INVALID_ARG, "infer NULL desc");
    expect(cola_fwd_outer(&ok, 11, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL),
           COLA_ERR_INVALID_ARG, "bad outer act");
    /* groups */
    cola_group_desc g;
    memset(&g, 0, sizeof(g));
    g.T = 64; g.d_in = 32; g.n = 9; g.dtype = COLA_BF16; g.act = COLA_ACT_SILU;
    expect((int)cola_group_workspace_bytes(&g, 1), 0, "n > 8");
    g.n = 2; g.r[0] = 8; g.r[1] = 8; g.d_out[0] = 32; g.d_out[1] = 40;
    (void)cola_group_workspace_bytes(&g, 0);
    (void)cola_group_workspace_bytes(&g, 1);
    (void)cola_group_workspace_bytes(&g, 2);
    expect(cola_group_fwd(&g, FAKE, FAKE, NULL, NULL, FAKE, FAKE, FAKE, 1 << 20, NULL), COLA_ERR_INVALID_ARG,
           "group NULL arrays");
    /* dense */
    dense_desc dd = {64, 32, 24, 0, 0, COLA_BF16};
    (void)dense_workspace_bytes(&dd, 1);
    dd.d_in = 0;
    expect(dense_fwd(&dd, FAKE, FAKE, FAKE, FAKE, 1 << 20, NULL), COLA_ERR_BAD_SHAPE, "dense d_in = 0");
    /* block */
    for (int64_t h = 1; h < 40; h += 7) {
        cola_block_desc b = {2, 256, 512, 1376, h, 128, COLA_ACT_SILU, (int)(h & 1), 10000.0f, 1e-6f};
        (void)cola_block_saved_bytes(&b);
        (void)cola_block_workspace_bytes(&b, 0);
        (void)cola_block_workspace_bytes(&b, 1);
        size_t off;
        int64_t ld;
        for (int s = -1; s <= COLA_BLK_SLOTS; ++s) (void)cola_block_saved_slot(&b, s, &off, &ld);
    }
    cola_block_desc b = {2, 256, 512, 1376, 8, 128, COLA_ACT_SILU, 0, 10000.0f, 1e-6f};
    cola_block_weights w;
    void** wp = (void**)&w;
    for (unsigned i = 0; i < sizeof(w) / sizeof(void*); ++i) wp[i] = FAKE;
    expect(cola_block_fwd(&b, NULL, FAKE, FAKE, FAKE, 1 << 30, FAKE, 1 << 30, NULL), COLA_ERR_INVALID_ARG,
           "block NULL weights");
    expect(cola_block_fwd(&b, &w, (char*)FAKE + 4, FAKE, FAKE, (size_t)1 << 40, FAKE, (size_t)1 << 40, NULL),
           COLA_ERR_INVALID_ARG, "block misaligned input");
    expect(cola_block_bwd(&b, &w, FAKE, FAKE, 1, FAKE, FAKE, NULL, FAKE, 1, NULL), COLA_ERR_INVALID_ARG,
           "block NULL grads");
    b.heads = 16;
    expect(cola_block_fwd(&b, &w, FAKE, FAKE, FAKE, 1, FAKE, 1, NULL), COLA_ERR_UNSUPPORTED, "head dim 32");
    b.heads = 8; b.rope_base = -1.0f;
    expect(cola_block_fwd(&b, &w, FAKE, FAKE, FAKE, 1, FAKE, 1, NULL), COLA_ERR_INVALID_ARG, "bad rope base");
    /* options, names, status text */
    expect(cola_set_option(99, 0), COLA_ERR_INVALID_ARG, "unknown option");
    expect(cola_set_option(COLA_OPT_WGRAD_PAIR, 5), COLA_ERR_INVALID_ARG, "option value");
    for (int k = -2; k < COLA_KC_COUNT + 2; ++k) (void)cola_kernel_name(k);
    for (int s = -1; s < 9; ++s) (void)cola_strerror(s);
    int64_t n;
    double ms, fl, by;
    expect(cola_timing_read(-1, &n, &ms, &fl, &by), COLA_ERR_INVALID_ARG, "timing bad class");
    printf(failures ? "abi sanitizer driver: %d FAILED\n" : "abi sanitizer driver: ok%.0d\n", failures);
    return failures ? 1 : 0;
}
