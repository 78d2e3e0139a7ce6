// Internal declarations shared by the HIP sources of libbevpool.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bevpool.h"

namespace bevpool {

// Work partition of the forward pass.
//
// Cells with points are grouped into tiles along the camera rays. A cell's
// key is (camera, feature column / kKeyCols, depth bin / kKeyBins) of its
// lowest-id point. Cells with one key lie along a short bundle of
// neighbouring rays, so their points share few distinct feature rows; each
// row is reused about once per depth bin the bundle spends in the tile. A
// key group becomes one tile, unless it has more than kPointBudget points or
// kMaxTileCells cells. Then it is cut where its running point count crosses
// a multiple of kPointBudget / 2, around every cell with more than
// kPointBudget / 2 points, and every kMaxTileCells cells. So a tile holds
// at most kPointBudget points, except a tile that is one heavier cell.
// One workgroup serves each tile. It stages the tile's distinct feature
// rows in LDS once, and every point reads its row from there.
//
// The forward kernel runs kPersistentGroups workgroups of kPersistentWaves
// waves, one per CU. Each owns a contiguous run of tiles of about equal cost
// and a share of the cells without points, which it zeroes. A tile heavier
// than kPointBudget (one cell) gets an extra workgroup of its own.
constexpr int kWaveSize = 64;
constexpr int kWaves = 4;                                  // plan kernels, heavy tiles
constexpr int kBlock = kWaves * kWaveSize;
constexpr int kPersistentGroups = 256;
constexpr int kPersistentWaves = 8;
constexpr int kPersistentBlock = kPersistentWaves * kWaveSize;
constexpr int kKeyCols = 4;
constexpr int kKeyBins = 8;
constexpr int kPointBudget = 2048;
constexpr int kMaxTileCells = 256;
constexpr int kStagePerThread = kPointBudget / kBlock;     // 8
constexpr int kFeatureLdsBytes = 56 * 1024;                // staged feature slab
static_assert(kPointBudget % kBlock == 0, "staging loop assumes whole rounds");

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
    int32_t n_cells, n_nonempty, max_per_cell, n_tiles, n_rows, n_empty, n_heavy;
    // canonical association (exported)
    int32_t *cell_of_point;  // [n_points]
    int32_t *sorted_point;   // [n_points]: kept ids by (cell, id), then dropped ids
    int32_t *cell_start;     // [n_cells + 1]
    // forward work partition, all in tile order
    int32_t *tile_cell_begin;  // [n_tiles + 1] into tile_cells / comp_cell_start
    int32_t *tile_row_begin;   // [n_tiles + 1] into row_pix
    int32_t *tile_cells;       // [n_nonempty] cells with points, tile by tile, id order inside
    int32_t *comp_cell_start;  // [n_nonempty + 1] first point (in comp order) of each listed cell
    int32_t *empty_cells;      // [n_empty] cells without points, in id order
    int32_t *tile_hdr;         // [n_tiles][8]: cell begin, cells, point begin, points, row begin, rows
    int32_t *heavy_tiles;      // [n_heavy] tiles with more than kPointBudget points
    int32_t *group_tile_begin; // [kPersistentGroups + 1] tile run of each persistent workgroup
    int32_t *comp_point;       // [n_kept] point ids, tile by tile, cell by cell, id order
    int32_t *comp_row;         // [n_kept] the point's feature row, relative to its tile
    int32_t *row_pix;          // [n_rows] pixel (n*H*W + h*W + w) of each staged row
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
