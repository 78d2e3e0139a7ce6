/*
 * Runs every function of the CPU oracle (oracle/bevpool_oracle.c) on small
 * rigs, for a build with AddressSanitizer and UndefinedBehaviorSanitizer: an
 * out-of-bounds access, a use of freed memory, a signed overflow or a bad
 * shift aborts the program. The checks here are light (the oracle's pins
 * live in tests/test_oracle_pins.py): the kept-point count of the one-camera
 * rig whose cell map has a closed form (224 of 256 points), the count test
 * (P = F = 1 gives each cell its point count), and mass conservation.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct {
    int32_t n_cams, feat_h, feat_w, n_depth;
    double depth_min, depth_step, pixel_offset;
    int32_t nx, ny;
    double x_min, y_min, cell_x, cell_y;
    double z_min, z_cell;
} oracle_geometry;

int64_t oracle_cell_map(const double *, const double *, const oracle_geometry *, int32_t *);
void oracle_sort_by_cell(const int32_t *, int64_t, int32_t, int32_t *, int32_t *);
void oracle_pool(const float *, const float *, const int32_t *, const oracle_geometry *, int32_t,
                 int32_t, float *, double *, double *);
void oracle_pool_reduce(const float *, const float *, const int32_t *, const oracle_geometry *,
                        int32_t, int32_t, int32_t, double *);
void oracle_backward(const float *, const float *, const float *, const int32_t *,
                     const oracle_geometry *, int32_t, int32_t, double *, double *);
void oracle_set_threads(int);

#define CHECK(c, ...) do { if (!(c)) { printf("FAIL: " __VA_ARGS__); printf("\n"); return 1; } } while (0)

static uint64_t state = 0x2545F4914F6CDD1Dull;
static float unit(void) {   /* xorshift64*, top 24 bits -> [0, 1) */
    state ^= state >> 12; state ^= state << 25; state ^= state >> 27;
    return (float)((state * 0x2545F4914F6CDD1Dull) >> 40) / 16777216.0f;
}

static int run(const double *intr, const double *extr, const oracle_geometry *g, int64_t expect_kept) {
    const int64_t np = (int64_t)g->n_cams * g->n_depth * g->feat_h * g->feat_w;
    const int64_t npix = (int64_t)g->n_cams * g->feat_h * g->feat_w;
    const int32_t nc = g->nx * g->ny;
    const int B = 2, C = 5;
    int32_t *cop = malloc(sizeof(int32_t) * np), *sp = malloc(sizeof(int32_t) * np);
    int32_t *cs = malloc(sizeof(int32_t) * (nc + 1));
    float *P = malloc(sizeof(float) * B * np), *F = malloc(sizeof(float) * B * npix * C);
    float *G = malloc(sizeof(float) * B * nc * C), *out = malloc(sizeof(float) * B * nc * C);
    double *o64 = malloc(sizeof(double) * B * nc * C), *a64 = malloc(sizeof(double) * B * nc * C);
    double *dP = malloc(sizeof(double) * B * np), *dF = malloc(sizeof(double) * B * npix * C);
    const int64_t kept = oracle_cell_map(intr, extr, g, cop);
    if (expect_kept >= 0) CHECK(kept == expect_kept, "kept %lld, expected %lld", (long long)kept, (long long)expect_kept);
    oracle_sort_by_cell(cop, np, nc, sp, cs);
    CHECK(cs[0] == 0 && cs[nc] == kept, "interval table ends");
    /* count test: P = F = 1, one channel */
    for (int64_t i = 0; i < np; ++i) P[i] = 1.0f;
    for (int64_t i = 0; i < npix; ++i) F[i] = 1.0f;
    oracle_pool(P, F, cop, g, 1, 1, out, o64, a64);
    for (int32_t c = 0; c < nc; ++c) CHECK(out[c] == (float)(cs[c + 1] - cs[c]), "count of cell %d", c);
    /* random inputs through every function */
    for (int64_t i = 0; i < B * np; ++i) P[i] = unit();
    for (int64_t i = 0; i < B * npix * C; ++i) F[i] = 2.0f * unit() - 1.0f;
    for (int64_t i = 0; i < B * nc * C; ++i) G[i] = 2.0f * unit() - 1.0f;
    oracle_pool(P, F, cop, g, B, C, out, o64, a64);
    const int64_t HW = (int64_t)g->feat_h * g->feat_w;
    for (int b = 0; b < B; ++b)
        for (int c = 0; c < C; ++c) {
            double mass = 0.0, got = 0.0, scale = 0.0;
            for (int64_t p = 0; p < np; ++p)
                if (cop[p] >= 0) {
                    const int64_t pix = (p / (g->n_depth * HW)) * HW + p % HW;
                    const double v = (double)P[b * np + p] * F[(b * npix + pix) * C + c];
                    mass += v;
                    scale += fabs(v);
                }
            for (int32_t k = 0; k < nc; ++k) got += o64[((int64_t)b * nc + k) * C + c];
            CHECK(fabs(got - mass) <= 1e-12 * (scale + 1.0), "mass of frame %d channel %d", b, c);
        }
    oracle_pool_reduce(P, F, cop, g, B, C, 1, o64);
    oracle_pool_reduce(P, F, cop, g, B, C, 2, o64);
    oracle_backward(P, F, G, cop, g, B, C, dP, dF);
    for (int64_t p = 0; p < np; ++p) if (cop[p] < 0) CHECK(dP[p] == 0.0, "dropped point gradient");
    free(cop); free(sp); free(cs); free(P); free(F); free(G); free(out); free(o64); free(a64);
    free(dP); free(dF);
    return 0;
}

int main(void) {
    oracle_set_threads(2);
    /* one camera at the origin looking along ego +x: closed-form cell map */
    const double intr1[4] = {4.0, 4.0, 4.0, 2.0};
    const double extr1[12] = {0, 0, 1, 0, -1, 0, 0, 0, 0, -1, 0, 0};
    const oracle_geometry g1 = {1, 4, 8, 8, 1.0, 1.0, 0.5, 16, 16, -8.0, -8.0, 1.0, 1.0, -10.0, 20.0};
    if (run(intr1, extr1, &g1, 224)) return 1;
    /* two cameras (the second turned 90 degrees), odd sizes, a coarse grid */
    const double intr2[8] = {5.0, 4.5, 3.5, 2.5, 6.0, 6.0, 3.5, 2.5};
    const double extr2[24] = {0, 0, 1, 0.2, -1, 0, 0, 0.1, 0, -1, 0, 1.5,
                              1, 0, 0, -0.1, 0, 0, 1, 0.3, 0, -1, 0, 1.5};
    const oracle_geometry g2 = {2, 5, 7, 9, 1.0, 0.75, 0.5, 11, 13, -6.0, -5.0, 1.1, 0.9, -2.0, 5.0};
    if (run(intr2, extr2, &g2, -1)) return 1;
    printf("PASS\n");
    return 0;
}
