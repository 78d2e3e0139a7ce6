// C ABI of libbevpool.so (declared in include/bevpool.h): argument checks,
// error reporting and plan ownership. Device work is in plan.hip and
// forward.hip.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <new>

#include "internal.h"

namespace {
thread_local char g_last_error[512] = "";

bool finite_all(const double *v, size_t n) {
    for (size_t i = 0; i < n; ++i)
        if (!isfinite(v[i])) return false;
    return true;
}

bool valid_plan(const bevpool_plan_t *plan) { return plan != nullptr && plan->magic == kPlanMagic; }

void free_plan(bevpool_plan_s *plan) {
    if (!plan) return;
    int prev = -1;
    (void)hipGetDevice(&prev);
    if (prev != plan->device) (void)hipSetDevice(plan->device);
    (void)hipFree(plan->cell_of_point);
    (void)hipFree(plan->sorted_point);
    (void)hipFree(plan->cell_start);
    (void)hipFree(plan->column_table);
    (void)hipFree(plan->generic_hdr);
    (void)hipFree(plan->generic_runs);
    (void)hipFree(plan->empty_cells);
    (void)hipFree(plan->multi_begin);
    (void)hipFree(plan->multi_cell);
    (void)hipFree(plan->multi_rows);
    (void)hipFree(plan->combo_cells);
    (void)hipFree(plan->combo_cols);
    (void)hipFree(plan->bwd_mixed);
    if (prev >= 0 && prev != plan->device) (void)hipSetDevice(prev);
    plan->magic = 0;
    delete plan;
}
}  // namespace

int bevpool_fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return code;
}

int bevpool_hip_fail(hipError_t err, const char *what) {
    return bevpool_fail(BEVPOOL_ERR_HIP, "HIP error %d (%s) in %s", int(err), hipGetErrorString(err),
                        what);
}

extern "C" {

const char *bevpool_last_error(void) { return g_last_error; }

int32_t bevpool_version(void) { return 200; }  // 0.2.0: bevpool_forward_ex

namespace {
// Sizes and parameters of a geometry (both plan constructors).
int check_geometry(const bevpool_geometry &g, int32_t nz = 1) {
    if (g.n_cams < 1 || g.feat_h < 1 || g.feat_w < 1 || g.n_depth < 1 || g.nx < 1 || g.ny < 1)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                            "sizes must be >= 1 (n_cams=%d feat_h=%d feat_w=%d n_depth=%d nx=%d ny=%d)",
                            g.n_cams, g.feat_h, g.feat_w, g.n_depth, g.nx, g.ny);
    const double params[] = {g.depth_min, g.depth_step, g.pixel_offset, g.x_min, g.y_min,
                             g.cell_x,    g.cell_y,     g.z_min,        g.z_cell};
    if (!finite_all(params, sizeof(params) / sizeof(params[0])))
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "geometry parameters must be finite");
    if (!(g.depth_step > 0.0) || !(g.cell_x > 0.0) || !(g.cell_y > 0.0) || !(g.z_cell > 0.0))
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                            "depth_step, cell_x, cell_y and z_cell must be positive");
    const int64_t np = int64_t(g.n_cams) * g.n_depth * g.feat_h * g.feat_w;
    if (np > int64_t(INT32_MAX))
        return bevpool_fail(BEVPOOL_ERR_OVERFLOW, "N*D*H*W = %lld points exceeds int32",
                            (long long)np);
    if (int64_t(g.nx) * g.ny * nz + 1 > int64_t(INT32_MAX))
        return bevpool_fail(BEVPOOL_ERR_OVERFLOW, "nx*ny*nz = %lld cells exceeds int32",
                            (long long)(int64_t(g.nx) * g.ny * nz));
    return BEVPOOL_OK;
}

int make_plan(const double *intrinsics, const double *extrinsics, const int32_t *host_cells,
              const bevpool_geometry &g, int32_t nz, void *hip_stream, bevpool_plan_t **out_plan) {
    bevpool_plan_s *plan = new (std::nothrow) bevpool_plan_s();
    if (!plan) return bevpool_fail(BEVPOOL_ERR_OOM, "host allocation of the plan failed");
    memset(plan, 0, sizeof(*plan));
    plan->magic = kPlanMagic;
    plan->geom = g;
    hipError_t e = hipGetDevice(&plan->device);
    if (e != hipSuccess) {
        delete plan;
        return bevpool_hip_fail(e, "hipGetDevice");
    }
    plan->nz = nz;
    const int rc = bevpool_build_plan(intrinsics, extrinsics, host_cells, g, nz,
                                      hipStream_t(hip_stream), plan);
    if (rc != BEVPOOL_OK) {
        free_plan(plan);
        return rc;
    }
    *out_plan = plan;
    return BEVPOOL_OK;
}
}  // namespace

int bevpool_plan_slabs(const double *intrinsics, const double *extrinsics,
                       const bevpool_geometry *geom, int32_t nz, void *hip_stream,
                       bevpool_plan_t **out_plan) {
    g_last_error[0] = '\0';
    if (!out_plan) return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "out_plan is NULL");
    *out_plan = nullptr;
    if (!intrinsics || !extrinsics || !geom)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "intrinsics, extrinsics and geom must be non-NULL");
    if (nz < 1) return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "nz=%d must be >= 1", nz);
    const bevpool_geometry &g = *geom;
    int rc = check_geometry(g, nz);
    if (rc != BEVPOOL_OK) return rc;
    if (!finite_all(intrinsics, size_t(4) * g.n_cams) || !finite_all(extrinsics, size_t(12) * g.n_cams))
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "calibration values must be finite");
    for (int n = 0; n < g.n_cams; ++n)
        if (intrinsics[4 * n] == 0.0 || intrinsics[4 * n + 1] == 0.0)
            return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "camera %d has a zero focal length", n);
    return make_plan(intrinsics, extrinsics, nullptr, g, nz, hip_stream, out_plan);
}

int bevpool_plan(const double *intrinsics, const double *extrinsics, const bevpool_geometry *geom,
                 void *hip_stream, bevpool_plan_t **out_plan) {
    return bevpool_plan_slabs(intrinsics, extrinsics, geom, 1, hip_stream, out_plan);
}

int bevpool_associate_noalloc(const double *intrinsics, const double *extrinsics,
                              const bevpool_geometry *geom, int32_t *cell_of_point,
                              int32_t *sorted_point, int32_t *cell_start, void *hip_stream) {
    g_last_error[0] = '\0';
    if (!intrinsics || !extrinsics || !geom || !cell_of_point || !sorted_point || !cell_start)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                            "intrinsics, extrinsics, geom and the three outputs must be non-NULL");
    const bevpool_geometry &g = *geom;
    int rc = check_geometry(g);
    if (rc != BEVPOOL_OK) return rc;
    if (!finite_all(intrinsics, size_t(4) * g.n_cams) || !finite_all(extrinsics, size_t(12) * g.n_cams))
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "calibration values must be finite");
    for (int n = 0; n < g.n_cams; ++n)
        if (intrinsics[4 * n] == 0.0 || intrinsics[4 * n + 1] == 0.0)
            return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "camera %d has a zero focal length", n);
    return bevpool_associate_into(intrinsics, extrinsics, g, cell_of_point, sorted_point, cell_start,
                                  hipStream_t(hip_stream));
}

int bevpool_plan_import(const int32_t *cell_of_point, const bevpool_geometry *geom,
                        void *hip_stream, bevpool_plan_t **out_plan) {
    g_last_error[0] = '\0';
    if (!out_plan) return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "out_plan is NULL");
    *out_plan = nullptr;
    if (!cell_of_point || !geom)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "cell_of_point and geom must be non-NULL");
    const bevpool_geometry &g = *geom;
    int rc = check_geometry(g);
    if (rc != BEVPOOL_OK) return rc;
    const int64_t np = int64_t(g.n_cams) * g.n_depth * g.feat_h * g.feat_w;
    const int32_t n_cells = g.nx * g.ny;
    for (int64_t p = 0; p < np; ++p)
        if (cell_of_point[p] < -1 || cell_of_point[p] >= n_cells)
            return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                                "cell_of_point[%lld] = %d is neither -1 nor a cell below %d",
                                (long long)p, cell_of_point[p], n_cells);
    return make_plan(nullptr, nullptr, cell_of_point, g, 1, hip_stream, out_plan);
}

namespace {
// The plan's arrays live on the device it was built on; a call on another
// device would read that memory through another device's stream.
int check_device(const bevpool_plan_t *plan) {
    int cur = -1;
    BEVPOOL_HIP(hipGetDevice(&cur));
    if (cur != plan->device)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                            "the plan was built on device %d but the current device is %d",
                            plan->device, cur);
    return BEVPOOL_OK;
}

int forward_checked(const void *depth_prob, const void *cam_feat, const bevpool_plan_t *plan,
                    float *bev_out, int64_t out_row_stride, int32_t batch, int32_t channels,
                    int32_t dtype, int32_t reduce, void *hip_stream, void *start_event,
                    void *stop_event) {
    if (!valid_plan(plan)) return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "invalid plan handle");
    if (!depth_prob || !cam_feat || !bev_out)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                            "depth_prob, cam_feat and bev_out must be non-NULL");
    if (batch < 1 || channels < 1)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "batch=%d and channels=%d must be >= 1", batch,
                            channels);
    if (dtype != BEVPOOL_F32 && dtype != BEVPOOL_BF16 && dtype != BEVPOOL_F16)
        return bevpool_fail(BEVPOOL_ERR_UNSUPPORTED_DTYPE, "dtype %d is not F32, BF16 or F16", dtype);
    if (reduce != BEVPOOL_SUM && reduce != BEVPOOL_MEAN && reduce != BEVPOOL_MAX)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "reduce %d is not SUM, MEAN or MAX", reduce);
    if (out_row_stride < channels)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "out_row_stride=%lld is below channels=%d",
                            (long long)out_row_stride, channels);
    const int rc = check_device(plan);
    if (rc != BEVPOOL_OK) return rc;
    return bevpool_launch_forward(depth_prob, cam_feat, plan, bev_out, out_row_stride, batch,
                                  channels, dtype, reduce, hipStream_t(hip_stream),
                                  hipEvent_t(start_event), hipEvent_t(stop_event));
}
}  // namespace

int bevpool_forward(const void *depth_prob, const void *cam_feat, const bevpool_plan_t *plan,
                    float *bev_out, int32_t batch, int32_t channels, int32_t dtype,
                    void *hip_stream) {
    return forward_checked(depth_prob, cam_feat, plan, bev_out, channels, batch, channels, dtype,
                           BEVPOOL_SUM, hip_stream, nullptr, nullptr);
}

int bevpool_forward_ex(const void *depth_prob, const void *cam_feat, const bevpool_plan_t *plan,
                       float *bev_out, int64_t out_row_stride, int32_t batch, int32_t channels,
                       int32_t dtype, int32_t reduce, void *hip_stream) {
    return forward_checked(depth_prob, cam_feat, plan, bev_out, out_row_stride, batch, channels,
                           dtype, reduce, hip_stream, nullptr, nullptr);
}

int bevpool_forward_timed(const void *depth_prob, const void *cam_feat, const bevpool_plan_t *plan,
                          float *bev_out, int32_t batch, int32_t channels, int32_t dtype,
                          void *hip_stream, void *start_event, void *stop_event) {
    return forward_checked(depth_prob, cam_feat, plan, bev_out, channels, batch, channels, dtype,
                           BEVPOOL_SUM, hip_stream, start_event, stop_event);
}

int bevpool_backward(const float *grad_out, const void *depth_prob, const void *cam_feat,
                     const bevpool_plan_t *plan, float *grad_depth, float *grad_feat,
                     int32_t batch, int32_t channels, int32_t dtype, void *hip_stream) {
    if (!valid_plan(plan)) return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "invalid plan handle");
    if (!grad_out || !depth_prob || !cam_feat)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                            "grad_out, depth_prob and cam_feat must be non-NULL");
    if (!grad_depth && !grad_feat)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "grad_depth and grad_feat are both NULL");
    if (batch < 1 || channels < 1)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "batch=%d and channels=%d must be >= 1", batch,
                            channels);
    if (dtype != BEVPOOL_F32 && dtype != BEVPOOL_BF16 && dtype != BEVPOOL_F16)
        return bevpool_fail(BEVPOOL_ERR_UNSUPPORTED_DTYPE, "dtype %d is not F32, BF16 or F16", dtype);
    const int rc = check_device(plan);
    if (rc != BEVPOOL_OK) return rc;
    return bevpool_launch_backward(grad_out, depth_prob, cam_feat, plan, grad_depth, grad_feat,
                                   batch, channels, dtype, hipStream_t(hip_stream));
}

int bevpool_to_nchw(const float *bev_nhwc, int64_t in_row_stride, float *bev_nchw, int32_t batch,
                    int32_t ny, int32_t nx, int32_t channels, void *hip_stream) {
    if (!bev_nhwc || !bev_nchw)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "bev_nhwc and bev_nchw must be non-NULL");
    if (batch < 1 || ny < 1 || nx < 1 || channels < 1)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                            "batch=%d, ny=%d, nx=%d and channels=%d must be >= 1", batch, ny, nx,
                            channels);
    if (in_row_stride < channels)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "in_row_stride=%lld is below channels=%d",
                            (long long)in_row_stride, channels);
    return bevpool_launch_to_nchw(bev_nhwc, in_row_stride, bev_nchw, batch, ny, nx, channels,
                                  hipStream_t(hip_stream));
}

int bevpool_plan_info_get(const bevpool_plan_t *plan, bevpool_plan_info *info) {
    if (!valid_plan(plan)) return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "invalid plan handle");
    if (!info) return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "info is NULL");
    info->n_points = plan->n_points;
    info->n_kept = plan->n_kept;
    info->n_cells = plan->n_cells;
    info->n_nonempty = plan->n_nonempty;
    info->max_per_cell = plan->max_per_cell;
    info->n_column = plan->n_column;
    info->n_generic = plan->n_generic;
    info->n_empty = plan->n_empty;
    info->n_runs = plan->n_runs;
    info->n_partials = plan->n_partials;
    info->n_multi = plan->n_multi;
    info->n_cams = plan->geom.n_cams;
    info->n_depth = plan->geom.n_depth;
    info->feat_h = plan->geom.feat_h;
    info->feat_w = plan->geom.feat_w;
    info->nx = plan->geom.nx;
    info->ny = plan->geom.ny;
    info->nz = plan->nz;
    info->n_planes = plan->n_planes;
    return BEVPOOL_OK;
}

int bevpool_plan_export(const bevpool_plan_t *plan, int32_t *cell_of_point, int32_t *sorted_point,
                        int32_t *cell_start) {
    if (!valid_plan(plan)) return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "invalid plan handle");
    if (cell_of_point)
        BEVPOOL_HIP(hipMemcpy(cell_of_point, plan->cell_of_point,
                              sizeof(int32_t) * size_t(plan->n_points), hipMemcpyDeviceToHost));
    if (sorted_point)
        BEVPOOL_HIP(hipMemcpy(sorted_point, plan->sorted_point,
                              sizeof(int32_t) * size_t(plan->n_kept), hipMemcpyDeviceToHost));
    if (cell_start)
        BEVPOOL_HIP(hipMemcpy(cell_start, plan->cell_start,
                              sizeof(int32_t) * (size_t(plan->n_cells) + 1), hipMemcpyDeviceToHost));
    return BEVPOOL_OK;
}

void bevpool_plan_destroy(bevpool_plan_t *plan) {
    if (!valid_plan(plan)) return;
    free_plan(plan);
}

}  // extern "C"
