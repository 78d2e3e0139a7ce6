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
// The points are split over column items of kColDepth depth bins x
// kColWidth pixel columns of one camera. A cell is "column-served" when
// all its points come from clean combos inside one item. Such a cell is
// computed by that item's workgroup: the workgroup reads each feature row
// (n, h, w) of its columns once and applies it to the kColDepth depth bins
// held in registers. A cell fed by a single combo is stored from
// registers; a cell fed by several combos of the item is summed through
// LDS. Every other cell with points is "generic": its points are gathered
// in runs of consecutive depth bins of one pixel. A generic cell gets one
// wave, or a whole workgroup when it has more than kGenHeavy points. Cells
// without points are zeroed by workgroups of their own.
constexpr int kWaveSize = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kWaves * kWaveSize;      // plan kernels and the forward kernel
constexpr int kGroupLanes = 16;                 // lanes per pixel column (one DPP row)
constexpr int kColDepth = 8;
constexpr int kColWidth = kBlock / kGroupLanes; // 16 columns per item
constexpr int kGenHeavy = 256;
constexpr int kSliceChannels = 80;              // channels per pass (LDS partials)

// Column-table entry flags (second word: h_lo | h_hi << 16 | flags).
constexpr uint32_t kComboMulti = 1u << 31;      // the cell has other combos
constexpr uint32_t kComboOwner = 1u << 30;      // first combo of a multi cell
constexpr int kMaxFeatH = 1 << 14;              // rows must fit the 15-bit fields

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
    int64_t n_points, n_kept;
    int32_t n_cells, n_nonempty, max_per_cell;
    int32_t n_column, n_generic, n_generic_heavy, n_runs, n_empty;
    // canonical association (exported)
    int32_t *cell_of_point;  // [n_points]
    int32_t *sorted_point;   // [n_points]: kept ids by (cell, id), then dropped ids
    int32_t *cell_start;     // [n_cells + 1]
    // forward work partition
    int2 *column_table;      // [N][D][W]: {cell or -1, h_lo | h_hi << 16 | flags}
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
int bevpool_build_plan(const double *intrinsics, const double *extrinsics,
                       const bevpool_geometry &g, hipStream_t stream,
                       bevpool_plan_s *plan);
int bevpool_launch_forward(const void *P, const void *F, const bevpool_plan_s *plan,
                           float *out, int32_t batch, int32_t channels,
                           int32_t dtype, hipStream_t stream);
