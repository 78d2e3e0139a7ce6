// Internal declarations shared by the HIP sources of libbevpool.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bevpool.h"

namespace bevpool {

// Work partition of the forward pass.
//
// A frustum point is (camera n, depth bin d, pixel row h, pixel column w).
// A "combo" is one (n, d, w): a column of H points on one depth plane. A
// combo is clean when all its kept points lie in one cell and their rows
// form one range h_lo..h_hi-1. A level camera makes almost every combo
// clean, since its rows then differ only in height.
//
// A cell whose points all come from clean combos is "column-served". The
// forward pass reads each feature row (n, h, w) once per block of
// kColDepth depth bins and applies it to all of them, with the sums of the
// block's combos held in registers (column items of kColDepth x
// kColWidth combos of one camera). A cell fed by one combo is stored from
// registers. A cell fed by several combos (near the rig a cell spans
// several pixel columns) gets one partial-sum slot per combo; slot s is the
// output row of the s-th empty cell, which is free until zeroed. A second
// kernel adds the slots of each such cell in slot order and then zeroes the
// borrowed rows. (A grid with fewer empty cells than slots serves these
// cells generically instead.) Every other cell
// with points is "generic": its points are gathered in runs of consecutive
// depth bins of one pixel, by one wave, or by a whole workgroup when it has
// more than kGenHeavy points. Cells without points are zeroed by
// workgroups of their own.
constexpr int kWaveSize = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kWaves * kWaveSize;      // plan kernels, combine kernel
constexpr int kFwdWaves = 2;
constexpr int kFwdBlock = kFwdWaves * kWaveSize;  // forward kernel
constexpr int kGroupLanes = 16;                 // lanes per pixel column
constexpr int kColDepth = 8;
constexpr int kColWidth = kFwdBlock / kGroupLanes;  // 8 columns per item
constexpr int kGenHeavy = 256;
constexpr int kSliceChannels = 128;             // channels per forward pass, at most
constexpr int kBwdSliceChannels = 80;           // channels per backward pass
constexpr int kBwdBlockCols = 8;                // pixel columns of a backward block
constexpr int kCombineInline = 8;               // borrowed rows listed with each multi-combo cell

// Column-table entry: {cell (single-combo cell) or borrowed row of its
// partial slot (multi), h_lo | h_hi << 16 | kComboMulti}.
constexpr uint32_t kComboMulti = 1u << 31;
constexpr int kMaxFeatH = 1 << 14;              // rows must fit the 15-bit fields
constexpr int kMaxSeg = 4;                      // row segments of a combo served by column items

// Unsigned division by a run-time constant through a multiply-high, after
// Granlund and Montgomery, "Division by invariant integers using
// multiplication" (PLDI 1994), Sec. 4: with l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1, n / d = (mulhi(m, n) + n) >> l for
// every n < 2^31 (the sum then stays below 2^32).
struct FastDiv {
    uint32_t d, m, l;
};

inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while ((uint64_t(1) << l) < d) ++l;
    const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
    return FastDiv{d, uint32_t(m), l};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
    return (__umulhi(f.m, n) + n) >> f.l;
}

}  // namespace bevpool

struct bevpool_plan_s {
    uint32_t magic;
    int device;
    bevpool_geometry geom;
    int32_t nz;              // stacked z slabs; cell id (iy * nx + ix) * nz + iz
    int64_t n_points, n_kept;
    int32_t n_cells, n_nonempty, max_per_cell;
    int32_t n_column, n_generic, n_generic_heavy, n_runs, n_empty;
    int32_t n_partials, n_multi;
    // canonical association (exported)
    int32_t *cell_of_point;  // [n_points]
    int32_t *sorted_point;   // [n_points]: kept ids by (cell, id), then dropped ids
    int32_t *cell_start;     // [n_cells + 1]
    // forward work partition
    int2 *column_table;      // [N][D][W]: {cell or borrowed row or -1, h_lo | h_hi << 16 | flags}
    int32_t *combo_cells;    // [N][D][W]: cell of a clean combo, -1 none kept, -2 not clean
    int2 *combo_cols;        // [N][W][D]: {cell, kept rows h_lo | h_hi << 16} of a clean combo, else {-1, 0}
    // backward work split: per camera and block of kBwdBlockCols pixel
    // columns, 1 when a combo of the block is not clean (such blocks take
    // the per-row kernel, the others the matrix-core kernel)
    int32_t *bwd_mixed;      // [N][ceil(W / kBwdBlockCols)]
    int32_t n_bwd_blocks, n_bwd_mixed;
    int32_t *multi_begin;    // [n_multi + 1]: first partial slot of each multi-combo cell
    int32_t *multi_cell;     // [n_multi]
    int32_t *multi_rows;     // [n_multi][kCombineInline]: borrowed rows of the first slots, or -1
    int32_t n_planes;        // segment planes of the column table in use (1 for a level rig)
    int4 *generic_hdr;       // [n_generic]: {cell, first run, runs, points}, most points first
    int4 *generic_runs;      // [n_runs]: {first point id, pixel, depth bins, 0}
    int32_t *empty_cells;    // [n_empty] cells without points, ascending
};

constexpr uint32_t kPlanMagic = 0xB3F9001Du;

// Error reporting (bevpool.hip).
int bevpool_fail(int code, const char *fmt, ...);
int bevpool_hip_fail(hipError_t err, const char *what);

#define BEVPOOL_HIP(call)                                      \
    do {                                                       \
        hipError_t e_ = (call);                                \
        if (e_ != hipSuccess) return bevpool_hip_fail(e_, #call); \
    } while (0)

// Plan building (plan.hip) and the forward pass (forward.hip).
// Plan building (plan.hip): from the calibration, or, when host_cells is
// not null, from a stored cell map (validated by the caller).
int bevpool_build_plan(const double *intrinsics, const double *extrinsics,
                       const int32_t *host_cells, const bevpool_geometry &g, int32_t nz,
                       hipStream_t stream, bevpool_plan_s *plan);
int bevpool_launch_backward(const float *G, const void *P, const void *F,
                            const bevpool_plan_s *plan, float *dP, float *dF, int32_t batch,
                            int32_t channels, int32_t dtype, hipStream_t stream);
int bevpool_launch_to_nchw(const float *in, int64_t in_row_stride, float *out, int32_t batch,
                           int32_t ny, int32_t nx, int32_t channels, hipStream_t stream);
// The association alone into caller buffers, with no allocation (plan.hip):
// temporaries in a fixed device array of kAssocScratchTotal bytes per device.
constexpr int64_t kAssocMaxPoints = int64_t(1) << 22;
constexpr int kAssocMaxCams = 16;
constexpr size_t kAssocScratchTotal = 54529280;   // 52 MiB
int bevpool_associate_into(const double *intrinsics, const double *extrinsics,
                           const bevpool_geometry &g, int32_t *cell_of_point,
                           int32_t *sorted_point, int32_t *cell_start, hipStream_t stream);
int bevpool_launch_forward(const void *P, const void *F, const bevpool_plan_s *plan,
                           float *out, int64_t ldo, int32_t batch, int32_t channels,
                           int32_t dtype, int32_t reduce, hipStream_t stream,
                           hipEvent_t start, hipEvent_t stop);
