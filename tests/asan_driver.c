/* Host-side driver for an AddressSanitizer pass over the library's host code: every
 * argument check, the buffer registry and the host-only helpers, called with real
 * heap arrays sized exactly (so any out-of-bounds host access is reported) and with
 * fake device addresses that every call must reject before anything is enqueued. Built
 * and run by tests/test_asan_host.py on a machine without a GPU. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../include/bc.h"

static int failures = 0;
#define EXPECT(cond) do { if (!(cond)) { fprintf(stderr, "line %d: %s (%s)\n", __LINE__, #cond, bc_last_error()); ++failures; } } while (0)

#define FAKE(a) ((void *)(uintptr_t)(a))

static bc_tensor T(int n, int c, int h, int w, int dt, int lay)
{
    bc_tensor t = {n, c, h, w, dt, lay};
    return t;
}

int main(void)
{
    /* status text for every code and beyond */
    for (int s = 0; s < 14; ++s) EXPECT(bc_status_str(s) != NULL && strlen(bc_status_str(s)) > 0);
    EXPECT(bc_abi_version() == BC_ABI_VERSION);

    /* host helpers on exact-size heap arrays */
    const int cout = 5, cin = 3, k = 3, per = cin * k * k;
    float *w = malloc(sizeof(float) * cout * per), *b = malloc(sizeof(float) * cout);
    float *g = malloc(sizeof(float) * cout), *be = malloc(sizeof(float) * cout);
    float *mu = malloc(sizeof(float) * cout), *var = malloc(sizeof(float) * cout);
    float *wo = malloc(sizeof(float) * cout * per), *bo = malloc(sizeof(float) * cout);
    for (int i = 0; i < cout * per; ++i) w[i] = (float)(i % 7) - 3.0f;
    for (int i = 0; i < cout; ++i) { b[i] = 0.5f; g[i] = 1.5f; be[i] = -0.25f; mu[i] = 0.1f; var[i] = 2.0f; }
    EXPECT(bc_fold_bn(w, cout, per, b, g, be, mu, var, 1e-5f, wo, bo) == BC_OK);
    EXPECT(fabsf(bo[0] - (-0.25f + (0.5f - 0.1f) * 1.5f / sqrtf(2.0f + 1e-5f))) < 1e-5f);
    EXPECT(bc_fold_bn(w, cout, per, NULL, g, be, mu, var, 1e-5f, wo, bo) == BC_OK);
    EXPECT(bc_fold_bn(NULL, cout, per, NULL, g, be, mu, var, 1e-5f, wo, bo) == BC_ERR_NULL);
    uint16_t *h16 = malloc(sizeof(uint16_t) * cout * per);
    float *h32 = malloc(sizeof(float) * cout * per);
    EXPECT(bc_repack_weights(w, cout, cin, k, k, BC_BF16, h16) == BC_OK);
    EXPECT(bc_repack_weights(w, cout, cin, k, k, BC_F16, h16) == BC_OK);
    EXPECT(bc_repack_weights(w, cout, cin, k, k, BC_F32, h32) == BC_OK);
    EXPECT(h32[1] == w[1 * k * k]);                       /* [co][i][j][ci] <- [co][ci][i][j] */
    EXPECT(bc_repack_weights(w, cout, cin, k, k, 7, h16) == BC_ERR_DTYPE);
    EXPECT(bc_repack_weights(w, 0, cin, k, k, BC_BF16, h16) == BC_ERR_SHAPE);

    /* buffer registry */
    bc_buffer h1 = NULL, h2 = NULL;
    EXPECT(bc_buffer_register(FAKE(0x10000000), T(1, 64, 32, 32, BC_BF16, BC_NHWC), &h1) == BC_OK);
    EXPECT(bc_buffer_register(FAKE(0x10000040), T(1, 64, 32, 32, BC_BF16, BC_NHWC), &h2) == BC_ERR_ALIAS);
    EXPECT(bc_buffer_is_valid(h1) == 0);
    EXPECT(bc_buffer_mark_written(h1, 1) == BC_OK && bc_buffer_is_valid(h1) == 1);
    EXPECT(bc_buffer_invalidate(h1) == BC_OK && bc_buffer_is_valid(h1) == 0);
    EXPECT(bc_buffer_release(h1) == BC_OK);
    EXPECT(bc_buffer_register(NULL, T(1, 64, 32, 32, BC_BF16, BC_NHWC), &h2) == BC_ERR_NULL);

    /* argument checks of the device entry points (fake addresses, all rejected) */
    bc_grid grid = {8, 16};
    bc_conv c3 = {3, 3, 1, 1, 1};
    void *in = FAKE(0x20000000), *wt = FAKE(0x30000000), *out = FAKE(0x40000000);
    int32_t *idx = FAKE(0x50000000), *cnt = FAKE(0x60000000);
    bc_tensor ti = T(1, 64, 64, 128, BC_BF16, BC_NHWC);
    EXPECT(bc_build_block_index(NULL, 1, grid, idx, 128, cnt, NULL, NULL) == BC_ERR_NULL);
    EXPECT(bc_build_block_index(FAKE(0x70000000), 1, grid, idx, 127, cnt, NULL, NULL) == BC_ERR_CAPACITY);
    EXPECT(bc_sparse_conv2d(&c3, NULL, ti, wt, NULL, NULL, out, ti, grid, idx, cnt, 128, NULL) == BC_ERR_NULL);
    EXPECT(bc_sparse_conv2d(&c3, in, ti, wt, NULL, NULL, out, T(1, 64, 32, 128, BC_BF16, BC_NHWC), grid, idx, cnt, 128, NULL) == BC_ERR_SHAPE);
    EXPECT(bc_sparse_conv2d(&c3, in, ti, wt, NULL, NULL, FAKE(0x20000010), ti, grid, idx, cnt, 128, NULL) == BC_ERR_ALIAS);
    EXPECT(bc_sparse_conv2d_noalloc(&c3, in, ti, wt, NULL, NULL, out, ti, (bc_grid){7, 16}, idx, cnt, 128, NULL) == BC_ERR_NOT_DIVISIBLE);
    EXPECT(bc_sparse_conv2d_noalloc(&c3, in, T(1, 512, 64, 128, BC_BF16, BC_NHWC), wt, NULL, NULL, out,
                                    T(1, 1024, 64, 128, BC_BF16, BC_NHWC), grid, idx, cnt, 128, NULL) == BC_ERR_CAPACITY);
    bc_conv_call ca = {{1, 1, 1, 0, 0}, in, ti, wt, NULL, NULL, out, T(1, 256, 64, 128, BC_BF16, BC_NHWC)};
    bc_conv_call cb = ca;
    EXPECT(bc_sparse_conv2d_pair(&ca, NULL, grid, idx, cnt, 128, NULL) == BC_ERR_NULL);
    EXPECT(bc_sparse_conv2d_pair(&ca, &cb, grid, idx, cnt, 128, NULL) == BC_ERR_ALIAS);   /* same output */
    bc_spp_geom sg = {4, 32, {8, 4, 2, 1}, {16, 8, 4, 2}};
    EXPECT(bc_sparse_spp(in, T(1, 128, 32, 64, BC_BF16, BC_NHWC), &sg, wt, NULL, FAKE(0x78000000), out,
                         T(1, 255, 32, 64, BC_BF16, BC_NHWC), grid, idx, cnt, 128, NULL) == BC_ERR_SHAPE);
    sg.levels = 9;
    EXPECT(bc_sparse_spp(in, T(1, 128, 32, 64, BC_BF16, BC_NHWC), &sg, wt, NULL, FAKE(0x78000000), out,
                         T(1, 256, 32, 64, BC_BF16, BC_NHWC), grid, idx, cnt, 128, NULL) == BC_ERR_SHAPE);
    bc_conv pool = {3, 3, 2, 1, 0};
    EXPECT(bc_sparse_maxpool2d(&pool, in, T(1, 64, 64, 128, BC_BF16, BC_NHWC), out, T(1, 32, 32, 64, BC_BF16, BC_NHWC),
                               grid, idx, cnt, 128, NULL) == BC_ERR_SHAPE);
    EXPECT(bc_gather_halo(in, ti, grid, &c3, 0.0f, idx, cnt, 127, out, NULL) == BC_ERR_CAPACITY);
    EXPECT(bc_scatter_blocks(NULL, idx, cnt, 128, grid, out, ti, NULL) == BC_ERR_NULL);
    EXPECT(bc_sparse_upsample_add(in, T(1, 64, 16, 32, BC_BF16, BC_NHWC), NULL, out, T(1, 64, 31, 64, BC_BF16, BC_NHWC),
                                  grid, 0, idx, cnt, 128, NULL) != BC_OK);
    EXPECT(bc_sample_execution_grid(NULL, 1, grid, 1, 0, FAKE(0x70000000), idx, 128, cnt, NULL, NULL) == BC_ERR_NULL);
    EXPECT(bc_rmsprop_step(NULL, NULL, NULL, 16, 1e-4f, 0.99f, 1e-8f, 0.0f, NULL, BC_BF16, NULL) == BC_ERR_NULL);
    EXPECT(bc_last_error() != NULL);

    free(w); free(b); free(g); free(be); free(mu); free(var); free(wo); free(bo); free(h16); free(h32);
    if (failures) {
        fprintf(stderr, "%d failures\n", failures);
        return 1;
    }
    printf("asan driver ok\n");
    return 0;
}
