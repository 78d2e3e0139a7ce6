/*
 * bevpool.h -- C ABI of libbevpool.so: camera-to-BEV pooling on MI355X (gfx950).
 *
 * The operation is the BEV pooling step of BEVFusion (arXiv 2205.13542,
 * Sec. III-B). Each camera feature pixel is lifted to D points along its
 * camera ray, and each point carries its depth probability times the pixel's
 * feature vector. The points are quantised to an r x r BEV grid and flattened
 * along z (first paragraph). All points of a cell are summed, or averaged,
 * or their maximum is taken (the "Interval Reduction" paragraph names sum,
 * mean and max; bevpool_forward sums, bevpool_forward_ex does all three).
 *
 * The point-to-cell association depends only on the calibration, so it is
 * computed once per rig ("Precomputation" paragraph). That is bevpool_plan.
 * Every frame then runs bevpool_forward.
 *
 * Conventions that hold for every call:
 *  - Return value: BEVPOOL_OK (0) on success, a negative BEVPOOL_ERR_* code
 *    otherwise. bevpool_last_error() then gives a message. No C++ exception
 *    and no abort crosses this boundary.
 *  - Pointers marked "host" are ordinary CPU memory. Pointers marked "device"
 *    are HIP device memory on the current device.
 *  - The caller owns every input and output buffer. The library owns the
 *    plan and its device buffers until bevpool_plan_destroy.
 *  - hip_stream is a hipStream_t passed as void*; NULL is the null stream.
 */
#ifndef BEVPOOL_H
#define BEVPOOL_H

#include <stdint.h>

/* Exported symbols stay visible when the library is built with hidden
 * default visibility. */
#ifndef BEVPOOL_API
#if defined(__GNUC__)
#define BEVPOOL_API __attribute__((visibility("default")))
#else
#define BEVPOOL_API
#endif
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define BEVPOOL_OK 0
#define BEVPOOL_ERR_INVALID_ARG (-1)       /* null pointer, non-positive size, non-finite or zero parameter */
#define BEVPOOL_ERR_SHAPE_MISMATCH (-2)    /* a size does not agree with the plan */
#define BEVPOOL_ERR_UNSUPPORTED_DTYPE (-3) /* dtype not one of bevpool_dtype */
#define BEVPOOL_ERR_OVERFLOW (-4)          /* a point, pixel or output index would not fit in int32 */
#define BEVPOOL_ERR_OOM (-5)               /* device allocation failed */
#define BEVPOOL_ERR_HIP (-6)               /* a HIP runtime call failed (message has the HIP error) */

/* Element type of depth_prob and cam_feat. Accumulation and output are fp32. */
typedef enum { BEVPOOL_F32 = 0, BEVPOOL_BF16 = 1, BEVPOOL_F16 = 2 } bevpool_dtype;

/* Aggregation of a cell's points (the "Interval Reduction" paragraph of
 * Sec. III-B names mean, max and sum as symmetric functions to use). A cell
 * without points gets 0 in every mode. */
typedef enum { BEVPOOL_SUM = 0, BEVPOOL_MEAN = 1, BEVPOOL_MAX = 2 } bevpool_reduce;

/*
 * Frustum and BEV grid (Sec. III-B, first paragraph: N cameras, an H x W
 * feature map, D depth bins, grid step r, z flattened).
 *  - Depth bin k lies at camera-frame depth depth_min + k * depth_step,
 *    k in [0, n_depth). The paper's typical workload uses 1 m + 0.5 m * k,
 *    118 bins (Sec. III-B footnote).
 *  - Feature pixel (h, w) sits at image point (w + pixel_offset, h + pixel_offset)
 *    in feature-grid pixels.
 *  - Cells: ix = floor((x - x_min) / cell_x) in [0, nx) and
 *    iy = floor((y - y_min) / cell_y) in [0, ny), in the ego frame. One z slab:
 *    a point is kept only if floor((z - z_min) / z_cell) == 0.
 *  - Cell id = iy * nx + ix. Points outside the grid or the slab are dropped.
 */
typedef struct {
    int32_t n_cams, feat_h, feat_w, n_depth; /* N, H, W, D */
    double depth_min, depth_step;            /* depth of bin k = depth_min + k * depth_step */
    double pixel_offset;                     /* usually 0.5 (pixel centres) */
    int32_t nx, ny;                          /* cells along ego x and ego y */
    double x_min, y_min, cell_x, cell_y;     /* grid origin and cell sides, metres */
    double z_min, z_cell;                    /* the single z slab [z_min, z_min + z_cell) */
} bevpool_geometry;

/* Opaque plan: the camera-fixed point-to-cell association on the device. */
typedef struct bevpool_plan_s bevpool_plan_t;

/*
 * Build the plan ("Precomputation" paragraph of Sec. III-B).
 *  intrinsics: host double[n_cams][4] = {fx, fy, cx, cy}, in feature-grid pixels.
 *  extrinsics: host double[n_cams][12] = row-major [R | t], camera to ego:
 *              p_ego = R p_cam + t. Camera axes are x right, y down, z forward.
 *  geom:       host; copied.
 *  hip_stream: stream on which the plan kernels run.
 *  out_plan:   receives the new plan; on failure *out_plan is set to NULL.
 *
 * The frustum point with camera n, depth bin d and pixel (h, w) has id
 * p = ((n * D + d) * H + h) * W + w. Its camera-frame position is
 * depth * ((u - cx) / fx, (v - cy) / fy, 1). That position is mapped to the
 * ego frame and quantised. Everything is evaluated in IEEE double in a fixed
 * order with no fused multiply-add. The resulting cell ids match a plain CPU
 * evaluation of the same expressions bit for bit.
 *
 * The plan holds four things:
 *  - cell_of_point: each point's cell, or -1 if dropped;
 *  - sorted_point: the kept points ordered by cell, ties broken by point id;
 *  - cell_start: the interval table, so cell c owns
 *    sorted_point[cell_start[c] .. cell_start[c+1]);
 *  - a work partition used by bevpool_forward.
 *
 * Allocates device memory and synchronises hip_stream before returning.
 * The calibration arrays may be freed as soon as the call returns.
 * Errors: INVALID_ARG (null pointer, a size < 1, a non-finite value, a zero
 * focal length, a non-positive step or cell side), OVERFLOW (N*D*H*W or
 * nx*ny + 1 does not fit in int32), OOM, HIP.
 */
BEVPOOL_API int bevpool_plan(const double *intrinsics, const double *extrinsics,
                 const bevpool_geometry *geom, void *hip_stream,
                 bevpool_plan_t **out_plan);

/*
 * A plan over nz >= 1 stacked z slabs (Sec. III-B, first paragraph: the
 * lifted points are quantised on the grid and the features flattened along
 * z). z is quantised like x and y: iz = floor((z - z_min) / z_cell), and a
 * point is kept when 0 <= iz < nz (geom's z_cell is one slab's height). The
 * cell id is (iy * nx + ix) * nz + iz, so the plan has nx * ny * nz cells
 * and a forward map [batch][ny][nx][nz][channels] is the slabs' features
 * concatenated along channels, [batch][ny][nx][nz * channels], from one
 * forward call that reads the inputs once. nz = 1 is bevpool_plan.
 * Arguments, ownership and errors are those of bevpool_plan, plus
 * INVALID_ARG for nz < 1 and OVERFLOW when nx * ny * nz + 1 does not fit in
 * int32. bevpool_plan_import rebuilds single-slab plans only.
 */
BEVPOOL_API int bevpool_plan_slabs(const double *intrinsics, const double *extrinsics,
                       const bevpool_geometry *geom, int32_t nz, void *hip_stream,
                       bevpool_plan_t **out_plan);

/*
 * Pool one batch of frames with a plan (Sec. III-B: lift P x F, sum each
 * cell's points; "Interval Reduction": each cell's sum is written once).
 *
 *  depth_prob: device [batch][N][D][H][W] of dtype.
 *  cam_feat:   device [batch][N][H][W][channels] of dtype.
 *  bev_out:    device float [batch][n_cells][channels]: [batch][ny][nx][channels]
 *              for a plan of one z slab, [batch][ny][nx][nz * channels] for
 *              a plan of nz slabs (bevpool_plan_slabs). Every element is
 *              overwritten, and cells with no kept point are set to 0.
 *  batch in 1..65535, channels >= 1. N, D, H, W, nx and ny come from the
 *  plan; the caller's buffers must have those sizes (the library cannot see
 *  them).
 *
 * out[b][cell][c] = sum over kept points p of cell of
 * depth_prob[b][p] * cam_feat[b][pixel(p)][c]. The sum is accumulated in fp32
 * in an order fixed by the plan, so repeated calls give bitwise equal
 * results. No atomics touch bev_out. A cell fed by several (camera, depth
 * bin, pixel column) combos is summed in two steps: the combos' partial sums
 * are parked in rows of bev_out that belong to empty cells, then added in a
 * fixed order by a second kernel, which also zeroes those rows.
 *
 * Inputs must be finite; non-finite inputs give unspecified output.
 * Asynchronous on hip_stream: no host synchronisation, no allocation.
 * Inputs must not overlap bev_out. Buffers need only element alignment;
 * 16-byte aligned bev_out with channels % 4 == 0 zeroes empty rows with
 * 16-byte stores.
 * A plan is not modified by the forward pass and may be used from several
 * streams at once (with distinct output buffers).
 * Errors: INVALID_ARG (null pointer or a bad plan handle, batch outside
 * 1..65535, channels < 1, the current device not the one the plan was
 * built on), UNSUPPORTED_DTYPE, OVERFLOW (one frame's
 * depth_prob, cam_feat or bev_out reaches 2 GiB), HIP (launch failure).
 */
BEVPOOL_API int bevpool_forward(const void *depth_prob, const void *cam_feat,
                    const bevpool_plan_t *plan, float *bev_out,
                    int32_t batch, int32_t channels, int32_t dtype,
                    void *hip_stream);

/*
 * bevpool_forward with a choice of aggregation and a strided output.
 *  reduce:         a bevpool_reduce. SUM is bevpool_forward's sum. MEAN
 *                  divides each cell's fp32 sum by its number of kept points.
 *                  MAX takes, per channel, the largest fp32 product P * F over
 *                  the cell's kept points (exact: no sum is involved).
 *  out_row_stride: floats from one cell's row of bev_out to the next
 *                  (>= channels). The call writes floats [0, channels) of
 *                  each row and no other element of bev_out, so several
 *                  calls can fill disjoint channel ranges of one map: with
 *                  nz z slabs (one plan per slab, each slab's z_min raised by
 *                  z_cell), slab iz writes at bev_out + iz * channels with
 *                  out_row_stride = nz * channels, which flattens the slabs
 *                  along z by concatenating their channels (Sec. III-B, first
 *                  paragraph). Frame b starts at bev_out + b * ny * nx *
 *                  out_row_stride.
 * Other arguments, ownership, asynchrony and determinism are those of
 * bevpool_forward. Errors: those of bevpool_forward, and INVALID_ARG for an
 * unknown reduce or out_row_stride < channels; OVERFLOW when ny * nx *
 * out_row_stride floats reach 2 GiB.
 */
BEVPOOL_API int bevpool_forward_ex(const void *depth_prob, const void *cam_feat,
                       const bevpool_plan_t *plan, float *bev_out, int64_t out_row_stride,
                       int32_t batch, int32_t channels, int32_t dtype, int32_t reduce,
                       void *hip_stream);

/*
 * bevpool_forward (the per-frame pooling of Sec. III-B, first paragraph and
 * "Interval Reduction") with kernel-boundary timing, for measurement: start_event
 * and stop_event (hipEvent_t handles created by the caller; either may be
 * NULL) are recorded by the first and the last kernel dispatch of the
 * forward pass itself, so hipEventElapsedTime(start, stop) is the GPU time
 * of the forward pass without the queue gaps that events recorded as
 * separate stream entries add (several microseconds on MI355X). Arguments,
 * results and errors are otherwise those of bevpool_forward.
 */
BEVPOOL_API int bevpool_forward_timed(const void *depth_prob, const void *cam_feat,
                          const bevpool_plan_t *plan, float *bev_out,
                          int32_t batch, int32_t channels, int32_t dtype,
                          void *hip_stream, void *start_event, void *stop_event);

/*
 * Gradients of bevpool_forward, for training (the pooling of Sec. III-B is a
 * layer of a model trained end to end; it is bilinear in P and F). For each frame b, with
 * grad_out = d loss / d bev_out:
 *   grad_depth[b][p] = sum_c cam_feat[b][pixel(p)][c] * grad_out[b][cell(p)][c]
 *                      for a kept point p, 0 for a dropped one;
 *   grad_feat[b][pixel][c] = sum over the pixel's kept points p of
 *                      depth_prob[b][p] * grad_out[b][cell(p)][c]  (0 if none).
 *
 *  grad_out:   device float [batch][n_cells][channels] (the forward's map).
 *  depth_prob, cam_feat: the forward's inputs, device, of dtype.
 *  grad_depth: device float [batch][N][D][H][W], overwritten; NULL to skip.
 *  grad_feat:  device float [batch][N][H][W][channels], overwritten; NULL to
 *              skip (not both NULL).
 * Sums are accumulated in fp32 in an order fixed by the plan, so repeated
 * calls give bitwise equal results; no atomics, no allocation, no scratch.
 * Asynchronous on hip_stream. Buffers must not overlap. A plan may be used
 * by several backward and forward calls at once on different streams.
 * Errors: INVALID_ARG (null pointer, a bad plan handle, both outputs NULL,
 * batch outside 1..65535, channels < 1, the current device not the plan's),
 * UNSUPPORTED_DTYPE, OVERFLOW (one
 * frame's tensor reaches 2 GiB), HIP (launch failure).
 */
BEVPOOL_API int bevpool_backward(const float *grad_out, const void *depth_prob,
                     const void *cam_feat, const bevpool_plan_t *plan, float *grad_depth,
                     float *grad_feat, int32_t batch, int32_t channels, int32_t dtype,
                     void *hip_stream);

/*
 * Channel-major copy of a BEV map, for a convolutional BEV encoder that reads
 * [B][C][ny][nx] planes (Sec. III-C: the fused BEV features go through a
 * convolutional encoder, and the fusion concatenates channel planes).
 *  bev_nhwc:  device float, frame b's cell (iy, ix) row at
 *             bev_nhwc + (b * ny * nx + iy * nx + ix) * in_row_stride;
 *             channels [0, channels) of each row are read.
 *  bev_nchw:  device float [batch][channels][ny][nx], overwritten.
 * Needs no plan. Asynchronous on hip_stream; the buffers must not overlap.
 * Errors: INVALID_ARG (null pointer, a size below 1, in_row_stride <
 * channels, batch above 65535, more than 65535 tiles of 128 channels),
 * OVERFLOW (in_row_stride or ny * nx reaches 2^31), HIP (launch failure).
 */
BEVPOOL_API int bevpool_to_nchw(const float *bev_nhwc, int64_t in_row_stride, float *bev_nchw,
                    int32_t batch, int32_t ny, int32_t nx, int32_t channels,
                    void *hip_stream);

/* Sizes of a plan. All counts are per frame. */
typedef struct {
    int64_t n_points;     /* N*D*H*W */
    int64_t n_kept;       /* points inside the grid and the z slab */
    int32_t n_cells;      /* nx*ny*nz */
    int32_t n_nonempty;   /* cells with at least one point */
    int32_t max_per_cell; /* largest interval */
    int32_t n_cams, n_depth, feat_h, feat_w, nx, ny;
    int32_t n_column;     /* cells fed by one (camera, depth bin, pixel column) */
    int32_t n_generic;    /* other cells with points */
    int32_t n_empty;      /* cells without points */
    int32_t n_runs;       /* gather runs of the generic cells */
    int32_t n_partials;   /* partial-sum slots of cells fed by several combos */
    int32_t n_multi;      /* cells with partial-sum slots */
    int32_t nz;           /* stacked z slabs (n_cells = nx * ny * nz) */
    int32_t n_planes;     /* column-table planes in use: the most row segments a
                             column-served combo has (1 for a level rig, one slab) */
} bevpool_plan_info;

/* Fill *info: the sizes of the association ("Precomputation" paragraph of
 * Sec. III-B) and of the forward's work partition. Host only, no device
 * work. Errors: INVALID_ARG (null pointer or a bad plan handle). */
BEVPOOL_API int bevpool_plan_info_get(const bevpool_plan_t *plan, bevpool_plan_info *info);

/*
 * Copy the plan's association to host arrays (the "Precomputation"
 * paragraph of Sec. III-B: every point's grid index, and the points sorted
 * by that index with their ranks, which "Interval Reduction" turns into
 * per-cell intervals): cell_of_point [n_points] (-1 for a dropped point),
 * sorted_point [n_kept] (kept point ids by cell, then id) and cell_start
 * [n_cells + 1] (cell c's points are sorted_point[cell_start[c] ..
 * cell_start[c+1]-1]). Any of them may be NULL to skip it; the caller owns
 * the host arrays. Synchronous (copies from the plan's device).
 * Errors: INVALID_ARG (bad plan handle), HIP (copy failure).
 */
BEVPOOL_API int bevpool_plan_export(const bevpool_plan_t *plan, int32_t *cell_of_point,
                        int32_t *sorted_point, int32_t *cell_start);

/*
 * A plan from a stored association, for callers that keep it (the
 * "Precomputation" paragraph of Sec. III-B: the association depends only on
 * the calibration, so it is computed once and reused). cell_of_point is
 * host int32 [n_points] as bevpool_plan_export writes it: the cell of every
 * point in point-id order, -1 for a dropped one. geom gives the sizes (the
 * projection parameters are not used). The sort, the interval table and the
 * work partition are rebuilt on the device; for a map exported from a plan
 * with the same sizes the result equals that plan. Synchronises hip_stream.
 * Errors: INVALID_ARG (null pointer, bad sizes, an entry outside
 * [-1, nx*ny)), OVERFLOW, OOM, HIP.
 */
BEVPOOL_API int bevpool_plan_import(const int32_t *cell_of_point, const bevpool_geometry *geom,
                        void *hip_stream, bevpool_plan_t **out_plan);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * association that bevpool_plan computes and bevpool_plan_export returns,
 * written into the caller's device buffers with no allocation. Use it where a
 * calibration changes per frame and a plan cannot be rebuilt.
 *  intrinsics, extrinsics, geom: as for bevpool_plan (host; read before the
 *              call returns, so they may be freed at once).
 *  cell_of_point: device int32 [n_points], overwritten: each point's cell, -1
 *              for a dropped one.
 *  sorted_point:  device int32 [n_points], overwritten: the kept point ids by
 *              (cell, id), then the dropped ids in ascending order.
 *  cell_start:    device int32 [nx*ny + 1], overwritten: cell c owns
 *              sorted_point[cell_start[c] .. cell_start[c+1]); cell_start[nx*ny]
 *              is the kept count.
 * The results equal bevpool_plan's bit for bit. Limits: at most 2^22
 * points and 16 cameras. The temporaries live in one fixed device array of
 * 52 MiB per device, held while the library is loaded and shared by every
 * call on that device: calls that overlap on one device (two streams, or two
 * host threads) race and must be serialised by the caller. Asynchronous and
 * stream-ordered on hip_stream: no host synchronisation, no allocation, no
 * host-to-device copy. Buffers must not overlap.
 * Errors: INVALID_ARG (null pointer, a size < 1, a non-finite value, a zero
 * focal length, more points or cameras than the limits), OVERFLOW, HIP.
 */
BEVPOOL_API int bevpool_associate_noalloc(const double *intrinsics, const double *extrinsics,
                              const bevpool_geometry *geom, int32_t *cell_of_point,
                              int32_t *sorted_point, int32_t *cell_start, void *hip_stream);

/* Free a plan and its device memory. NULL-safe. The plan must not be in use
 * by work still queued on a stream. */
BEVPOOL_API void bevpool_plan_destroy(bevpool_plan_t *plan);

/* Message for the last nonzero return on the calling thread ("" if none). */
BEVPOOL_API const char *bevpool_last_error(void);

/* Library version as major * 10000 + minor * 100 + patch. */
BEVPOOL_API int32_t bevpool_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BEVPOOL_H */
