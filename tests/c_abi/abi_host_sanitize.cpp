/*
 * The C ABI's host layer (paper_2205_13542_amd/csrc/bevpool.hip: argument
 * checks, error messages, plan ownership) built for the host alone with
 * AddressSanitizer and UndefinedBehaviorSanitizer and linked against stubs:
 * the device work (plan build, kernel launches) and the few HIP runtime calls
 * the layer makes are replaced by functions defined here, so every error path
 * runs without a GPU and the sanitizers see all of the layer's memory use.
 * Each call is checked for the documented return code (include/bevpool.h).
 */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "internal.h"

// ---------------------------------------------------------------- stubs
static int g_device = 0;          // what hipGetDevice reports
static int g_build_rc = BEVPOOL_OK;
static int g_launches = 0;

extern "C" {
hipError_t hipGetDevice(int *d) { *d = g_device; return hipSuccess; }
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipFree(void *) { return hipSuccess; }
hipError_t hipMemcpy(void *dst, const void *, size_t n, hipMemcpyKind) { memset(dst, 0, n); return hipSuccess; }
const char *hipGetErrorString(hipError_t) { return "stub error"; }
}

int bevpool_build_plan(const double *, const double *, const int32_t *, const bevpool_geometry &g,
                       int32_t nz, hipStream_t, bevpool_plan_s *plan) {
    if (g_build_rc != BEVPOOL_OK) return bevpool_fail(g_build_rc, "stub build failure");
    plan->n_points = int64_t(g.n_cams) * g.n_depth * g.feat_h * g.feat_w;
    plan->n_kept = plan->n_points / 2;
    plan->n_cells = g.nx * g.ny * nz;
    return BEVPOOL_OK;
}
int bevpool_launch_forward(const void *, const void *, const bevpool_plan_s *, float *, int64_t,
                           int32_t, int32_t, int32_t, int32_t, hipStream_t, hipEvent_t, hipEvent_t) {
    ++g_launches;
    return BEVPOOL_OK;
}
int bevpool_launch_backward(const float *, const void *, const void *, const bevpool_plan_s *,
                            float *, float *, int32_t, int32_t, int32_t, hipStream_t) {
    ++g_launches;
    return BEVPOOL_OK;
}
int bevpool_launch_to_nchw(const float *, int64_t, float *, int32_t, int32_t, int32_t, int32_t,
                           hipStream_t) {
    ++g_launches;
    return BEVPOOL_OK;
}
int bevpool_associate_into(const double *, const double *, const bevpool_geometry &, int32_t *,
                           int32_t *, int32_t *, hipStream_t) {
    ++g_launches;
    return BEVPOOL_OK;
}

// ---------------------------------------------------------------- checks
#define EXPECT(call, code)                                                                   \
    do {                                                                                     \
        const int rc_ = (call);                                                              \
        if (rc_ != (code)) {                                                                 \
            printf("FAIL line %d: %s returned %d, expected %d (%s)\n", __LINE__, #call, rc_, \
                   int(code), bevpool_last_error());                                         \
            return 1;                                                                        \
        }                                                                                    \
        if ((code) != BEVPOOL_OK && bevpool_last_error()[0] == '\0') {                       \
            printf("FAIL line %d: %s left no message\n", __LINE__, #call);                   \
            return 1;                                                                        \
        }                                                                                    \
    } while (0)

static bevpool_geometry tiny() {
    bevpool_geometry g;
    memset(&g, 0, sizeof(g));
    g.n_cams = 1; g.feat_h = 4; g.feat_w = 8; g.n_depth = 8;
    g.depth_min = 1.0; g.depth_step = 1.0; g.pixel_offset = 0.5;
    g.nx = 16; g.ny = 16; g.x_min = -8.0; g.y_min = -8.0; g.cell_x = 1.0; g.cell_y = 1.0;
    g.z_min = -10.0; g.z_cell = 20.0;
    return g;
}

int main() {
    const double intr[4] = {4.0, 4.0, 4.0, 2.0};
    const double extr[12] = {0, 0, 1, 0, -1, 0, 0, 0, 0, -1, 0, 0};
    bevpool_geometry g = tiny();
    bevpool_plan_t *plan = nullptr;
    if (bevpool_version() < 100) { printf("FAIL version\n"); return 1; }

    // plan: arguments and geometry
    EXPECT(bevpool_plan(intr, extr, &g, nullptr, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_plan(nullptr, extr, &g, nullptr, &plan), BEVPOOL_ERR_INVALID_ARG);
    if (plan) { printf("FAIL: a failed call left a plan\n"); return 1; }
    EXPECT(bevpool_plan(intr, extr, nullptr, nullptr, &plan), BEVPOOL_ERR_INVALID_ARG);
    { bevpool_geometry b = g; b.n_cams = 0; EXPECT(bevpool_plan(intr, extr, &b, nullptr, &plan), BEVPOOL_ERR_INVALID_ARG); }
    { bevpool_geometry b = g; b.depth_min = NAN; EXPECT(bevpool_plan(intr, extr, &b, nullptr, &plan), BEVPOOL_ERR_INVALID_ARG); }
    { bevpool_geometry b = g; b.cell_x = 0.0; EXPECT(bevpool_plan(intr, extr, &b, nullptr, &plan), BEVPOOL_ERR_INVALID_ARG); }
    { bevpool_geometry b = g; b.z_cell = -1.0; EXPECT(bevpool_plan(intr, extr, &b, nullptr, &plan), BEVPOOL_ERR_INVALID_ARG); }
    { bevpool_geometry b = g; b.n_depth = 1 << 20; b.feat_h = 1 << 12; EXPECT(bevpool_plan(intr, extr, &b, nullptr, &plan), BEVPOOL_ERR_OVERFLOW); }
    { bevpool_geometry b = g; b.nx = 1 << 16; b.ny = 1 << 16; EXPECT(bevpool_plan(intr, extr, &b, nullptr, &plan), BEVPOOL_ERR_OVERFLOW); }
    { const double z[4] = {0.0, 4.0, 4.0, 2.0}; EXPECT(bevpool_plan(z, extr, &g, nullptr, &plan), BEVPOOL_ERR_INVALID_ARG); }
    { double e[12]; memcpy(e, extr, sizeof(e)); e[5] = INFINITY; EXPECT(bevpool_plan(intr, e, &g, nullptr, &plan), BEVPOOL_ERR_INVALID_ARG); }
    // a failing device build frees the half-built plan and leaves none
    g_build_rc = BEVPOOL_ERR_OOM;
    EXPECT(bevpool_plan(intr, extr, &g, nullptr, &plan), BEVPOOL_ERR_OOM);
    if (plan) { printf("FAIL: a failed build left a plan\n"); return 1; }
    g_build_rc = BEVPOOL_OK;
    EXPECT(bevpool_plan(intr, extr, &g, nullptr, &plan), BEVPOOL_OK);

    // stacked z slabs: nz is checked, and the cell count includes it
    {
        bevpool_plan_t *sl = nullptr;
        EXPECT(bevpool_plan_slabs(intr, extr, &g, 0, nullptr, &sl), BEVPOOL_ERR_INVALID_ARG);
        EXPECT(bevpool_plan_slabs(intr, extr, &g, 1 << 24, nullptr, &sl), BEVPOOL_ERR_OVERFLOW);
        EXPECT(bevpool_plan_slabs(intr, extr, &g, 4, nullptr, &sl), BEVPOOL_OK);
        bevpool_plan_info si;
        EXPECT(bevpool_plan_info_get(sl, &si), BEVPOOL_OK);
        if (si.nz != 4 || si.n_cells != 16 * 16 * 4) { printf("FAIL slab info\n"); return 1; }
        bevpool_plan_destroy(sl);
    }

    // import: every entry is validated on the host
    {
        const int64_t np = 1 * 8 * 4 * 8;
        int32_t cells[np];
        for (int64_t p = 0; p < np; ++p) cells[p] = int32_t(p % 257) - 1;   // -1 .. 255
        bevpool_plan_t *imp = nullptr;
        EXPECT(bevpool_plan_import(cells, &g, nullptr, &imp), BEVPOOL_OK);
        bevpool_plan_destroy(imp);
        cells[77] = 256;
        EXPECT(bevpool_plan_import(cells, &g, nullptr, &imp), BEVPOOL_ERR_INVALID_ARG);
        cells[77] = -2;
        EXPECT(bevpool_plan_import(cells, &g, nullptr, &imp), BEVPOOL_ERR_INVALID_ARG);
        EXPECT(bevpool_plan_import(nullptr, &g, nullptr, &imp), BEVPOOL_ERR_INVALID_ARG);
    }

    // info and export
    bevpool_plan_info info;
    EXPECT(bevpool_plan_info_get(plan, &info), BEVPOOL_OK);
    if (info.n_points != 256 || info.n_cells != 256 || info.nz != 1) { printf("FAIL info\n"); return 1; }
    EXPECT(bevpool_plan_info_get(plan, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_plan_info_get(nullptr, &info), BEVPOOL_ERR_INVALID_ARG);
    {
        int32_t cop[256], sp[128], cs[257];
        EXPECT(bevpool_plan_export(plan, cop, sp, cs), BEVPOOL_OK);
        EXPECT(bevpool_plan_export(plan, nullptr, nullptr, nullptr), BEVPOOL_OK);
        EXPECT(bevpool_plan_export(nullptr, cop, sp, cs), BEVPOOL_ERR_INVALID_ARG);
    }

    // forward arguments (buffers are never touched by the stubs)
    float dummy[4];
    const void *P = dummy, *F = dummy;
    float *O = dummy;
    g_launches = 0;
    EXPECT(bevpool_forward(P, F, plan, O, 1, 8, BEVPOOL_F32, nullptr), BEVPOOL_OK);
    EXPECT(bevpool_forward(nullptr, F, plan, O, 1, 8, BEVPOOL_F32, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_forward(P, F, nullptr, O, 1, 8, BEVPOOL_F32, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_forward(P, F, plan, O, 0, 8, BEVPOOL_F32, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_forward(P, F, plan, O, 1, 0, BEVPOOL_F32, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_forward(P, F, plan, O, 1, 8, 7, nullptr), BEVPOOL_ERR_UNSUPPORTED_DTYPE);
    EXPECT(bevpool_forward_ex(P, F, plan, O, 7, 1, 8, BEVPOOL_F32, BEVPOOL_SUM, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_forward_ex(P, F, plan, O, 8, 1, 8, BEVPOOL_F32, 9, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_forward_ex(P, F, plan, O, 12, 1, 8, BEVPOOL_BF16, BEVPOOL_MAX, nullptr), BEVPOOL_OK);
    EXPECT(bevpool_forward_timed(P, F, plan, O, 1, 8, BEVPOOL_F16, nullptr, nullptr, nullptr), BEVPOOL_OK);
    // a plan from another device is refused before any launch
    g_device = 3;
    EXPECT(bevpool_forward(P, F, plan, O, 1, 8, BEVPOOL_F32, nullptr), BEVPOOL_ERR_INVALID_ARG);
    if (!strstr(bevpool_last_error(), "device")) { printf("FAIL device message\n"); return 1; }
    EXPECT(bevpool_backward(dummy, P, F, plan, dummy, dummy, 1, 8, BEVPOOL_F32, nullptr), BEVPOOL_ERR_INVALID_ARG);
    g_device = 0;
    if (g_launches != 3) { printf("FAIL: %d launches, expected 3\n", g_launches); return 1; }

    // backward and layout
    EXPECT(bevpool_backward(dummy, P, F, plan, dummy, nullptr, 1, 8, BEVPOOL_F32, nullptr), BEVPOOL_OK);
    EXPECT(bevpool_backward(dummy, P, F, plan, nullptr, nullptr, 1, 8, BEVPOOL_F32, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_backward(nullptr, P, F, plan, dummy, dummy, 1, 8, BEVPOOL_F32, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_backward(dummy, P, F, plan, dummy, dummy, 1, 8, 5, nullptr), BEVPOOL_ERR_UNSUPPORTED_DTYPE);
    EXPECT(bevpool_to_nchw(dummy, 8, dummy, 1, 16, 16, 8, nullptr), BEVPOOL_OK);
    EXPECT(bevpool_to_nchw(dummy, 4, dummy, 1, 16, 16, 8, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_to_nchw(nullptr, 8, dummy, 1, 16, 16, 8, nullptr), BEVPOOL_ERR_INVALID_ARG);
    EXPECT(bevpool_to_nchw(dummy, 8, dummy, 1, 0, 16, 8, nullptr), BEVPOOL_ERR_INVALID_ARG);

    // the association without allocation: argument checks before any launch
    {
        int32_t *d = reinterpret_cast<int32_t *>(dummy);
        const int before = g_launches;
        EXPECT(bevpool_associate_noalloc(intr, extr, &g, d, d, d, nullptr), BEVPOOL_OK);
        EXPECT(bevpool_associate_noalloc(nullptr, extr, &g, d, d, d, nullptr), BEVPOOL_ERR_INVALID_ARG);
        EXPECT(bevpool_associate_noalloc(intr, extr, &g, d, nullptr, d, nullptr), BEVPOOL_ERR_INVALID_ARG);
        bevpool_geometry b = g;
        b.cell_y = -1.0;
        EXPECT(bevpool_associate_noalloc(intr, extr, &b, d, d, d, nullptr), BEVPOOL_ERR_INVALID_ARG);
        const double z[4] = {4.0, 0.0, 4.0, 2.0};
        EXPECT(bevpool_associate_noalloc(z, extr, &g, d, d, d, nullptr), BEVPOOL_ERR_INVALID_ARG);
        if (g_launches != before + 1) { printf("FAIL: association launches\n"); return 1; }
    }

    // a message longer than the buffer is cut, not overrun
    {
        bevpool_geometry b = g;
        b.n_cams = -2147483647; b.feat_h = -2147483647; b.feat_w = -2147483647;
        b.n_depth = -2147483647; b.nx = -2147483647; b.ny = -2147483647;
        bevpool_plan_t *none = nullptr;
        EXPECT(bevpool_plan(intr, extr, &b, nullptr, &none), BEVPOOL_ERR_INVALID_ARG);
        if (strlen(bevpool_last_error()) >= 512) { printf("FAIL message length\n"); return 1; }
    }
    bevpool_plan_destroy(plan);
    bevpool_plan_destroy(nullptr);
    printf("PASS\n");
    return 0;
}
