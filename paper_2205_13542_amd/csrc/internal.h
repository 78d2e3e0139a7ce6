// Internal declarations shared by the HIP sources of libbevpool.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bevpool.h"

namespace bevpool {

// Work partition of the forward pass.
//
// A frustum point is (camera n, depth bin d, pixel row h, pixel column w). A
// "combo" is one (n, d, w): a column of H points on one depth plane. A combo
// is clean when its kept points lie in one cell and their rows form one
// range h_lo..h_hi-1. A level camera makes every combo clean, since its rows
// then differ only in height.
//
// A cell is "swept" when all its points come from clean combos of one camera
// and one depth bin, in consecutive pixel columns. On a level camera the
// points of one depth bin lie on a straight line of the ground plane, so a
// cell meets that line in one stretch of columns: every cell that only one
// camera sees is swept. The sum of a swept cell is the sum over its columns
// of the column sums S[d][w][:] = sum_h P[d][h][w] F[h][w][:], a small dense
// product per pixel column (depth bins x rows by rows x channels). The
// forward pass computes these products on the matrix cores, 16 depth bins
// by 16 channels at a time, walks each depth bin's columns in order and
// writes a cell when its last column has been added (the column table flags
// a cell's first and last column). One workgroup covers a camera's full
// width for 16 depth bins and 16 channels, so every swept cell is finished
// inside one workgroup; cells that straddle two waves' column ranges are
// completed through LDS.
//
// Every other cell with points (cells seen by two cameras, cells of tilted
// cameras) is "generic": its points are gathered in runs of consecutive
// depth bins of one pixel, by one wave, or by a whole workgroup when it has
// more than kGenHeavy points. Cells without points are zeroed. All of it runs
// in one launch, and every output row is written once.
constexpr int kWaveSize = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kWaves * kWaveSize;      // plan kernels
constexpr int kGenHeavy = 256;
constexpr int kSliceChannels = 128;             // channels per generic-cell pass, at most
constexpr int kBwdSliceChannels = 80;           // channels per backward pass

// Forward workgroups: kSweepWaves waves; a sweep workgroup takes
// kSweepDepths depth bins x kSweepChannels channels of one camera.
constexpr int kSweepWaves = 16;
constexpr int kSweepBlock = kSweepWaves * kWaveSize;
constexpr int kSweepDepths = 16;                // matrix-core tile: N (depth bins)
constexpr int kSweepChannels = 16;              // matrix-core tile: M (channels)
constexpr int kSweepMaxCols = 12;               // pixel columns per wave, at most
constexpr int kSweepPBuf = 12288;               // floats per LDS buffer of staged probabilities

// Column-table entry of a combo of a swept cell: {cell, h_lo | h_hi << 15 |
// kColFirst | kColLast}; {-1, 0} for any other combo.
constexpr uint32_t kColFirst = 1u << 30;        // first column of its cell
constexpr uint32_t kColLast = 1u << 31;         // last column of its cell
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
    int32_t n_multi;         // swept cells fed by several combos
    int32_t n_run_cells;     // generic cells gathered in runs (the first of generic_hdr)
    int32_t n_combo_cells;   // generic cells gathered combo by combo
    int32_t n_cc_combos;     // their combos
    int32_t sweep_ok;        // the camera width fits one sweep workgroup
    int32_t n_cus;           // compute units of the plan's device
    // canonical association (exported)
    int32_t *cell_of_point;  // [n_points]
    int32_t *sorted_point;   // [n_points]: kept ids by (cell, id), then dropped ids
    int32_t *cell_start;     // [n_cells + 1]
    // forward work partition
    int2 *column_table;      // [N][W][D]: {cell, h_lo | h_hi << 15 | flags} or {-1, 0}
    int32_t *combo_cells;    // [N][D][W]: cell of a clean combo, -1 none kept, -2 not clean
    int4 *generic_hdr;       // [n_run_cells]: {cell, first run, runs, points}, most points first
    int4 *cc_hdr;            // [n_combo_cells]: {cell, first combo entry, entries, points}
    int2 *cc_list;           // [n_cc_combos]: {combo (n * D + d) * W + w, h_lo | h_hi << 15}
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
// Rows of staged depth probabilities per pass of a sweep workgroup for a
// camera W columns wide and H rows high (a multiple of 4), or 0 when a row of
// that width does not fit (plan.hip).
int bevpool_sweep_rows(int32_t W, int32_t H);
int bevpool_build_plan(const double *intrinsics, const double *extrinsics,
                       const int32_t *host_cells, const bevpool_geometry &g,
                       hipStream_t stream, bevpool_plan_s *plan);
int bevpool_launch_backward(const float *G, const void *P, const void *F,
                            const bevpool_plan_s *plan, float *dP, float *dF, int32_t batch,
                            int32_t channels, int32_t dtype, hipStream_t stream);
int bevpool_launch_to_nchw(const float *in, int64_t in_row_stride, float *out, int32_t batch,
                           int32_t ny, int32_t nx, int32_t channels, hipStream_t stream);
int bevpool_launch_forward(const void *P, const void *F, const bevpool_plan_s *plan,
                           float *out, int64_t ldo, int32_t batch, int32_t channels,
                           int32_t dtype, int32_t reduce, hipStream_t stream,
                           hipEvent_t start, hipEvent_t stop);
