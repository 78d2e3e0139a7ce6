/*
 * C round trip through libbevpool.so: no Python between the caller and the
 * library. A small level ring rig, fp32 inputs from a fixed xorshift
 * stream, two frames. Checked against the CPU oracle (liboracle.so):
 *  - the plan's cell of every point equals the oracle's cell map exactly;
 *  - the pooled map is within 1e-4 * sqrt(points in the cell) of the
 *    oracle's fp64 sums, and empty cells are exactly 0;
 *  - bevpool_forward_ex's max into channels [4, 4 + C) of rows C + 8 floats
 *    apart equals the oracle's max rounded to float, and the other floats
 *    of the map keep their contents;
 *  - bevpool_to_nchw gives the planes of the summed map exactly;
 *  - bevpool_plan_import rebuilds the plan from the exported cell map, and
 *    its pooled map equals the first plan's bit for bit;
 *  - bevpool_backward's gradients are within 1e-4 sqrt(C) (dP) and
 *    1e-4 sqrt(kept bins) (dF) of the oracle's;
 *  - bad arguments return the documented error codes with a message.
 * Exit status 0 when every check passes; the first failure is printed.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "bevpool.h"

/* The oracle's C interface (oracle/bevpool_oracle.c), declared here: the
 * oracle ships no header, and this program is the only C caller. */
typedef struct {
    int32_t n_cams, feat_h, feat_w, n_depth;
    double depth_min, depth_step, pixel_offset;
    int32_t nx, ny;
    double x_min, y_min, cell_x, cell_y;
    double z_min, z_cell;
} oracle_geometry;
int64_t oracle_cell_map(const double *intrinsics, const double *extrinsics,
                        const oracle_geometry *g, int32_t *cell_of_point);
void oracle_pool(const float *P, const float *F, const int32_t *cell_of_point,
                 const oracle_geometry *g, int32_t batch, int32_t channels, float *out,
                 double *out64, double *abs64);
void oracle_pool_reduce(const float *P, const float *F, const int32_t *cell_of_point,
                        const oracle_geometry *g, int32_t batch, int32_t channels,
                        int32_t mode, double *out64);
void oracle_backward(const float *P, const float *F, const float *G,
                     const int32_t *cell_of_point, const oracle_geometry *g,
                     int32_t batch, int32_t channels, double *dP64, double *dF64);

#define FAIL(...)                          \
    do {                                   \
        fprintf(stderr, "FAIL: " __VA_ARGS__); \
        fprintf(stderr, "\n");             \
        return 1;                          \
    } while (0)

#define HIP_OK(x)                                                        \
    do {                                                                 \
        hipError_t e_ = (x);                                             \
        if (e_ != hipSuccess) FAIL("%s -> %s", #x, hipGetErrorString(e_)); \
    } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static float next_unit(void) { /* xorshift64*, top 24 bits -> [0, 1) */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (float)((rng_state * 0x2545F4914F6CDD1Dull) >> 40) / 16777216.0f;
}

int main(void) {
    enum { N = 4, H = 8, W = 16, D = 12, NX = 40, NY = 40, C = 20, B = 2 };
    const double PI = 3.14159265358979323846;
    double intr[N * 4], extr[N * 12];
    for (int n = 0; n < N; ++n) {
        /* camera n looks along yaw n * 90 degrees, 1 m from the origin,
         * 1.5 m up; camera axes x right, y down, z forward */
        const double t = n * PI / 2, c = cos(t), s = sin(t);
        const double R[9] = {s, 0, c, -c, 0, s, 0, -1, 0};   /* columns: right, down, forward */
        double *E = extr + 12 * n;
        for (int r = 0; r < 3; ++r) {
            for (int k = 0; k < 3; ++k) E[4 * r + k] = R[3 * r + k];
        }
        E[3] = c;
        E[7] = s;
        E[11] = 1.5;
        intr[4 * n + 0] = 8.0;
        intr[4 * n + 1] = 8.0;
        intr[4 * n + 2] = W / 2.0;
        intr[4 * n + 3] = H / 2.0;
    }
    bevpool_geometry g;
    memset(&g, 0, sizeof(g));
    g.n_cams = N;
    g.feat_h = H;
    g.feat_w = W;
    g.n_depth = D;
    g.depth_min = 1.0;
    g.depth_step = 0.75;
    g.pixel_offset = 0.5;
    g.nx = NX;
    g.ny = NY;
    g.x_min = -10.0;
    g.y_min = -10.0;
    g.cell_x = 0.5;
    g.cell_y = 0.5;
    g.z_min = -5.0;
    g.z_cell = 10.0;
    oracle_geometry og = {N, H, W, D, 1.0, 0.75, 0.5, NX, NY, -10.0, -10.0, 0.5, 0.5, -5.0, 10.0};

    const int64_t n_points = (int64_t)N * D * H * W, n_pix = (int64_t)N * H * W;
    const int64_t n_cells = (int64_t)NX * NY;
    float *P = malloc(sizeof(float) * B * n_points);
    float *F = malloc(sizeof(float) * B * n_pix * C);
    float *got = malloc(sizeof(float) * B * n_cells * C);
    float *ref = malloc(sizeof(float) * B * n_cells * C);
    double *ref64 = malloc(sizeof(double) * B * n_cells * C);
    double *abs64 = malloc(sizeof(double) * B * n_cells * C);
    int32_t *cop_lib = malloc(sizeof(int32_t) * n_points);
    int32_t *cop_ref = malloc(sizeof(int32_t) * n_points);
    int32_t *count = calloc(n_cells, sizeof(int32_t));
    if (!P || !F || !got || !ref || !ref64 || !abs64 || !cop_lib || !cop_ref || !count)
        FAIL("host allocation");
    for (int64_t i = 0; i < B * n_points; ++i) P[i] = next_unit();
    for (int64_t i = 0; i < B * n_pix * C; ++i) F[i] = 2.0f * next_unit() - 1.0f;

    /* plan: association bit-exact against the oracle */
    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));
    bevpool_plan_t *plan = NULL;
    if (bevpool_plan(intr, extr, &g, stream, &plan) != BEVPOOL_OK)
        FAIL("bevpool_plan: %s", bevpool_last_error());
    if (bevpool_plan_export(plan, cop_lib, NULL, NULL) != BEVPOOL_OK)
        FAIL("bevpool_plan_export: %s", bevpool_last_error());
    const int64_t kept = oracle_cell_map(intr, extr, &og, cop_ref);
    if (kept <= 0) FAIL("the rig keeps no point");
    for (int64_t p = 0; p < n_points; ++p) {
        if (cop_lib[p] != cop_ref[p]) FAIL("cell of point %lld: %d, oracle %d", (long long)p, cop_lib[p], cop_ref[p]);
        if (cop_ref[p] >= 0) ++count[cop_ref[p]];
    }
    bevpool_plan_info info;
    if (bevpool_plan_info_get(plan, &info) != BEVPOOL_OK || info.n_kept != kept)
        FAIL("plan info: n_kept %lld, oracle %lld", (long long)info.n_kept, (long long)kept);

    /* forward on two frames; output prefilled with NaN */
    void *dP, *dF, *dO;
    HIP_OK(hipMalloc(&dP, sizeof(float) * B * n_points));
    HIP_OK(hipMalloc(&dF, sizeof(float) * B * n_pix * C));
    HIP_OK(hipMalloc(&dO, sizeof(float) * B * n_cells * C));
    HIP_OK(hipMemcpy(dP, P, sizeof(float) * B * n_points, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dF, F, sizeof(float) * B * n_pix * C, hipMemcpyHostToDevice));
    HIP_OK(hipMemset(dO, 0xFF, sizeof(float) * B * n_cells * C));
    if (bevpool_forward(dP, dF, plan, (float *)dO, B, C, BEVPOOL_F32, stream) != BEVPOOL_OK)
        FAIL("bevpool_forward: %s", bevpool_last_error());
    HIP_OK(hipStreamSynchronize(stream));
    HIP_OK(hipMemcpy(got, dO, sizeof(float) * B * n_cells * C, hipMemcpyDeviceToHost));
    oracle_pool(P, F, cop_ref, &og, B, C, ref, ref64, abs64);
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t c = 0; c < n_cells; ++c) {
            const double bound = 1e-4 * sqrt(count[c] > 1 ? (double)count[c] : 1.0);
            for (int k = 0; k < C; ++k) {
                const int64_t i = (b * n_cells + c) * C + k;
                const double err = fabs((double)got[i] - ref64[i]);
                if (!(err <= bound) || (count[c] == 0 && got[i] != 0.0f))
                    FAIL("frame %lld cell %lld channel %d: %.9g, oracle %.9g (points %d)",
                         (long long)b, (long long)c, k, got[i], ref64[i], count[c]);
            }
        }
    }

    /* max into a channel block of a wider map (sentinel 7.0 elsewhere) */
    enum { LD = C + 8, OFF = 4 };
    float *wide = malloc(sizeof(float) * B * n_cells * LD);
    double *max64 = malloc(sizeof(double) * B * n_cells * C);
    float *planes = malloc(sizeof(float) * B * n_cells * C);
    if (!wide || !max64 || !planes) FAIL("host allocation");
    void *dW, *dN;
    HIP_OK(hipMalloc(&dW, sizeof(float) * B * n_cells * LD));
    HIP_OK(hipMalloc(&dN, sizeof(float) * B * n_cells * C));
    for (int64_t i = 0; i < B * n_cells * LD; ++i) wide[i] = 7.0f;
    HIP_OK(hipMemcpy(dW, wide, sizeof(float) * B * n_cells * LD, hipMemcpyHostToDevice));
    if (bevpool_forward_ex(dP, dF, plan, (float *)dW + OFF, LD, B, C, BEVPOOL_F32, BEVPOOL_MAX,
                           stream) != BEVPOOL_OK)
        FAIL("bevpool_forward_ex: %s", bevpool_last_error());
    HIP_OK(hipStreamSynchronize(stream));
    HIP_OK(hipMemcpy(wide, dW, sizeof(float) * B * n_cells * LD, hipMemcpyDeviceToHost));
    oracle_pool_reduce(P, F, cop_ref, &og, B, C, 2, max64);
    for (int64_t r = 0; r < B * n_cells; ++r) {
        for (int k = 0; k < LD; ++k) {
            const float v = wide[r * LD + k];
            if (k < OFF || k >= OFF + C) {
                if (v != 7.0f) FAIL("row %lld float %d outside the block changed to %.9g", (long long)r, k, v);
            } else if (v != (float)max64[r * C + (k - OFF)]) {
                FAIL("max row %lld channel %d: %.9g, oracle %.9g", (long long)r, k - OFF, v,
                     max64[r * C + (k - OFF)]);
            }
        }
    }

    /* channel planes of the summed map: a copy, so exact */
    if (bevpool_to_nchw((const float *)dO, C, (float *)dN, B, NY, NX, C, stream) != BEVPOOL_OK)
        FAIL("bevpool_to_nchw: %s", bevpool_last_error());
    HIP_OK(hipStreamSynchronize(stream));
    HIP_OK(hipMemcpy(planes, dN, sizeof(float) * B * n_cells * C, hipMemcpyDeviceToHost));
    for (int64_t b = 0; b < B; ++b)
        for (int k = 0; k < C; ++k)
            for (int64_t c = 0; c < n_cells; ++c)
                if (planes[(b * C + k) * n_cells + c] != got[(b * n_cells + c) * C + k])
                    FAIL("plane %d of frame %lld, cell %lld differs", k, (long long)b, (long long)c);

    /* the plan rebuilt from its exported cell map pools the same map */
    bevpool_plan_t *imported = NULL;
    if (bevpool_plan_import(cop_lib, &g, stream, &imported) != BEVPOOL_OK)
        FAIL("bevpool_plan_import: %s", bevpool_last_error());
    if (bevpool_forward(dP, dF, imported, (float *)dN, B, C, BEVPOOL_F32, stream) != BEVPOOL_OK)
        FAIL("bevpool_forward on the imported plan: %s", bevpool_last_error());
    HIP_OK(hipStreamSynchronize(stream));
    HIP_OK(hipMemcpy(planes, dN, sizeof(float) * B * n_cells * C, hipMemcpyDeviceToHost));
    if (memcmp(planes, got, sizeof(float) * B * n_cells * C) != 0)
        FAIL("the imported plan pools a different map");
    bevpool_plan_destroy(imported);

    /* gradients against the oracle's, for G = 1 + 0.01 * element index mod 7 */
    {
        float *G = malloc(sizeof(float) * B * n_cells * C);
        float *gdP = malloc(sizeof(float) * B * n_points);
        float *gdF = malloc(sizeof(float) * B * n_pix * C);
        double *rdP = malloc(sizeof(double) * B * n_points);
        double *rdF = malloc(sizeof(double) * B * n_pix * C);
        if (!G || !gdP || !gdF || !rdP || !rdF) FAIL("host allocation");
        for (int64_t i = 0; i < B * n_cells * C; ++i) G[i] = 1.0f + 0.01f * (float)(i % 7);
        void *dG, *ddP, *ddF;
        HIP_OK(hipMalloc(&dG, sizeof(float) * B * n_cells * C));
        HIP_OK(hipMalloc(&ddP, sizeof(float) * B * n_points));
        HIP_OK(hipMalloc(&ddF, sizeof(float) * B * n_pix * C));
        HIP_OK(hipMemcpy(dG, G, sizeof(float) * B * n_cells * C, hipMemcpyHostToDevice));
        if (bevpool_backward((const float *)dG, dP, dF, plan, (float *)ddP, (float *)ddF, B, C,
                             BEVPOOL_F32, stream) != BEVPOOL_OK)
            FAIL("bevpool_backward: %s", bevpool_last_error());
        HIP_OK(hipStreamSynchronize(stream));
        HIP_OK(hipMemcpy(gdP, ddP, sizeof(float) * B * n_points, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(gdF, ddF, sizeof(float) * B * n_pix * C, hipMemcpyDeviceToHost));
        oracle_backward(P, F, G, cop_ref, &og, B, C, rdP, rdF);
        for (int64_t i = 0; i < B * n_points; ++i)
            if (!(fabs((double)gdP[i] - rdP[i]) <= 1e-4 * sqrt((double)C)))
                FAIL("dP[%lld] = %.9g, oracle %.9g", (long long)i, gdP[i], rdP[i]);
        for (int64_t b = 0; b < B; ++b)
            for (int64_t pix = 0; pix < n_pix; ++pix) {
                const int64_t n = pix / (H * W), hw = pix % (H * W);
                int kept_bins = 0;
                for (int d = 0; d < D; ++d) kept_bins += cop_ref[(n * D + d) * H * W + hw] >= 0;
                const double bound = 1e-4 * sqrt(kept_bins > 1 ? (double)kept_bins : 1.0);
                for (int k = 0; k < C; ++k) {
                    const int64_t i = (b * n_pix + pix) * C + k;
                    if (!(fabs((double)gdF[i] - rdF[i]) <= bound))
                        FAIL("dF[%lld] = %.9g, oracle %.9g", (long long)i, gdF[i], rdF[i]);
                }
            }
        HIP_OK(hipFree(dG));
        HIP_OK(hipFree(ddP));
        HIP_OK(hipFree(ddF));
        free(G); free(gdP); free(gdF); free(rdP); free(rdF);
    }

    /* documented errors */
    if (bevpool_forward(dP, dF, plan, (float *)dO, 0, C, BEVPOOL_F32, stream) != BEVPOOL_ERR_INVALID_ARG ||
        bevpool_last_error()[0] == '\0')
        FAIL("batch 0 must be INVALID_ARG with a message");
    if (bevpool_forward(dP, dF, plan, (float *)dO, B, C, 7, stream) != BEVPOOL_ERR_UNSUPPORTED_DTYPE)
        FAIL("dtype 7 must be UNSUPPORTED_DTYPE");
    if (bevpool_forward_ex(dP, dF, plan, (float *)dO, C - 1, B, C, BEVPOOL_F32, BEVPOOL_SUM, stream) !=
        BEVPOOL_ERR_INVALID_ARG)
        FAIL("a row stride below the channel count must be INVALID_ARG");
    if (bevpool_forward_ex(dP, dF, plan, (float *)dO, C, B, C, BEVPOOL_F32, 9, stream) !=
        BEVPOOL_ERR_INVALID_ARG)
        FAIL("reduce 9 must be INVALID_ARG");
    if (bevpool_forward(NULL, dF, plan, (float *)dO, B, C, BEVPOOL_F32, stream) != BEVPOOL_ERR_INVALID_ARG)
        FAIL("a null input must be INVALID_ARG");
    bevpool_plan_t *bad = NULL;
    if (bevpool_plan(NULL, extr, &g, stream, &bad) != BEVPOOL_ERR_INVALID_ARG || bad != NULL)
        FAIL("null intrinsics must be INVALID_ARG and leave no plan");

    bevpool_plan_destroy(plan);
    HIP_OK(hipFree(dP));
    HIP_OK(hipFree(dF));
    HIP_OK(hipFree(dO));
    HIP_OK(hipFree(dW));
    HIP_OK(hipFree(dN));
    HIP_OK(hipStreamDestroy(stream));
    printf("PASS: %lld kept points, %d non-empty cells, %d frames x %d channels\n",
           (long long)kept, info.n_nonempty, B, C);
    free(P); free(F); free(got); free(ref); free(ref64); free(abs64);
    free(cop_lib); free(cop_ref); free(count); free(wide); free(max64); free(planes);
    return 0;
}
