// Internal declarations shared by the HIP sources of libbevpool.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bevpool.h"

namespace bevpool {

// Work partition of the forward pass. The cells are cut into tiles of
// consecutive cell ids, one workgroup per tile. A tile's "path length" is
// kCellWeight * cells + points. A new tile starts whenever that length
// crosses a multiple of kTilePath. A cell with more than kHeavyPoints points
// gets a tile of its own. A multi-cell tile therefore holds fewer than
// kTilePath + kHeavyPoints points, all staged in LDS at once. Heavier
// single-cell tiles are staged in rounds of kStagePoints.
constexpr int kWaveSize = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kWaves * kWaveSize;
constexpr int kTilePath = 1024;
constexpr int kCellWeight = 1;
constexpr int kHeavyPoints = 512;
constexpr int kStagePoints = kTilePath + kHeavyPoints;        // 1536
constexpr int kMaxTileCells = kTilePath / kCellWeight + 1;    // 1025
constexpr int kStagePerThread = kStagePoints / kBlock;        // 6
static_assert(kStagePoints % kBlock == 0, "staging loop assumes whole rounds");

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
    int32_t n_cells, n_nonempty, max_per_cell, n_tiles;
    int32_t *cell_of_point;  // [n_points]
    int32_t *sorted_point;   // [n_points]: kept ids by (cell, id), then dropped ids
    int32_t *cell_start;     // [n_cells + 1]
    int32_t *tile_cell;      // [n_tiles + 1]
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
