// Plan building for BEV pooling: the camera-fixed point-to-cell association
// (BEVFusion, arXiv 2205.13542, Sec. III-B, "Precomputation" paragraph:
// compute each frustum point's 3-D coordinate and grid index once, sort the
// points by grid index and record their ranks).
//
// Kernels, in launch order:
//   k_project      one thread per point: camera ray -> ego frame -> cell id
//   k_radix_hist   } stable LSD radix sort of (cell, point id), 8-bit digits;
//   k_scan         } input in id order, so ties stay in id order
//   k_radix_scatter}
//   k_cell_start   interval table from the sorted keys
//   k_cell_stats   non-empty cells and the largest interval
//   k_cell_keys ... k_rows   ray-aligned work partition of the forward pass
//
// The geometry is evaluated in IEEE double with the file built without
// floating-point contraction, in one fixed expression order, so the cell ids
// equal those of any plain CPU evaluation of the same expressions.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <utility>

#include "internal.h"

#pragma clang fp contract(off)

namespace bevpool {
namespace {

constexpr int kSortItems = 8;                       // keys per thread per tile
constexpr int kSortTile = kBlock * kSortItems;      // 2048 keys per workgroup
constexpr int kWaveItems = kWaveSize * kSortItems;  // 512 keys per wave
constexpr int kScanBlock = 1024;
constexpr int kScanItems = 4;
static_assert(kBlock == 256, "one radix digit per thread");

struct ProjectArgs {
    const double *intr;  // [N][4]
    const double *extr;  // [N][12]
    bevpool_geometry g;
    FastDiv div_w, div_h, div_d;
    int32_t n_points, n_cells;
    int32_t *cell_of_point;
    uint32_t *keys;
    int32_t *vals;
};

// Sec. III-B, first paragraph: the pixel's ray at depth bin d, in the ego
// frame, quantised at the cell size; points outside the grid or the z slab
// are dropped. Sort key = cell id, or n_cells for a dropped point (last).
__global__ __launch_bounds__(kBlock) void k_project(ProjectArgs a) {
    const int32_t p = blockIdx.x * kBlock + threadIdx.x;
    if (p >= a.n_points) return;
    const bevpool_geometry &g = a.g;
    const uint32_t q_w = fdiv(uint32_t(p), a.div_w);
    const int w = p - int(q_w) * g.feat_w;
    const uint32_t q_h = fdiv(q_w, a.div_h);
    const int h = int(q_w) - int(q_h) * g.feat_h;
    const int n = int(fdiv(q_h, a.div_d));
    const int d = int(q_h) - n * g.n_depth;

    const double fx = a.intr[4 * n + 0], fy = a.intr[4 * n + 1];
    const double cx = a.intr[4 * n + 2], cy = a.intr[4 * n + 3];
    const double *E = a.extr + 12 * n;
    const double depth = g.depth_min + double(d) * g.depth_step;
    const double u = double(w) + g.pixel_offset;
    const double v = double(h) + g.pixel_offset;
    const double xc = depth * ((u - cx) / fx);
    const double yc = depth * ((v - cy) / fy);
    const double zc = depth;
    const double X = ((E[0] * xc + E[1] * yc) + E[2] * zc) + E[3];
    const double Y = ((E[4] * xc + E[5] * yc) + E[6] * zc) + E[7];
    const double Z = ((E[8] * xc + E[9] * yc) + E[10] * zc) + E[11];
    const double qx = floor((X - g.x_min) / g.cell_x);
    const double qy = floor((Y - g.y_min) / g.cell_y);
    const double qz = floor((Z - g.z_min) / g.z_cell);
    int32_t cell = -1;
    if (qx >= 0.0 && qx < double(g.nx) && qy >= 0.0 && qy < double(g.ny) && qz == 0.0)
        cell = int32_t(qy) * g.nx + int32_t(qx);
    a.cell_of_point[p] = cell;
    a.keys[p] = cell >= 0 ? uint32_t(cell) : uint32_t(a.n_cells);
    a.vals[p] = p;
}

// ---------------------------------------------------------------- scan

// Exclusive scan of one value per thread across the block; *total gets the
// block sum. Uses wave shuffles, then one LDS slot per wave.
template <int BLOCK>
__device__ __forceinline__ int block_exclusive_scan(int v, int *lds, int *total) {
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    int x = v;
#pragma unroll
    for (int off = 1; off < kWaveSize; off <<= 1) {
        const int y = __shfl_up(x, off, kWaveSize);
        if (lane >= off) x += y;
    }
    if (lane == kWaveSize - 1) lds[wave] = x;
    __syncthreads();
    int before = 0, sum = 0;
#pragma unroll
    for (int w = 0; w < BLOCK / kWaveSize; ++w) {
        const int s = lds[w];
        before += (w < wave) ? s : 0;
        sum += s;
    }
    __syncthreads();
    *total = sum;
    return before + x - v;
}

// In-place exclusive scan of data[0..n) by a single workgroup (plan-time
// only; sizes are at most a few million). *total receives the sum.
__global__ __launch_bounds__(kScanBlock) void k_scan(int32_t *data, int64_t n, int32_t *total) {
    __shared__ int lds[kScanBlock / kWaveSize];
    int carry = 0;
    for (int64_t base = 0; base < n; base += int64_t(kScanBlock) * kScanItems) {
        const int64_t i0 = base + int64_t(threadIdx.x) * kScanItems;
        int v[kScanItems];
        int local = 0;
#pragma unroll
        for (int k = 0; k < kScanItems; ++k) {
            v[k] = (i0 + k < n) ? data[i0 + k] : 0;
            local += v[k];
        }
        int blocksum;
        int run = carry + block_exclusive_scan<kScanBlock>(local, lds, &blocksum);
#pragma unroll
        for (int k = 0; k < kScanItems; ++k) {
            if (i0 + k < n) data[i0 + k] = run;
            run += v[k];
        }
        carry += blocksum;
    }
    if (threadIdx.x == 0) *total = carry;
}

// ---------------------------------------------------------------- radix sort

// Digit histogram of each 2048-key tile, stored digit-major:
// hist[digit * n_tiles + tile], so an exclusive scan of the whole array
// gives every (digit, tile) its first output slot in stable order.
__global__ __launch_bounds__(kBlock) void k_radix_hist(const uint32_t *keys, int32_t n,
                                                       int shift, int32_t *hist) {
    __shared__ int cnt[256];
    cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = int64_t(blockIdx.x) * kSortTile;
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = base + int64_t(k) * kBlock + threadIdx.x;
        if (i < n) atomicAdd(&cnt[(keys[i] >> shift) & 255u], 1);
    }
    __syncthreads();
    hist[int64_t(threadIdx.x) * gridDim.x + blockIdx.x] = cnt[threadIdx.x];
}

// Stable scatter. Wave w of a tile owns keys [w*512, (w+1)*512) of the tile
// and walks them 64 at a time in order. Within a step, a key's rank among
// equal digits comes from eight ballots (one per digit bit): lanes whose
// ballots agree on every bit hold the same digit. A per-wave LDS counter per
// digit carries ranks across steps. Per-wave counts are then prefixed across
// the waves and added to the scanned global offsets.
__global__ __launch_bounds__(kBlock) void k_radix_scatter(const uint32_t *keys_in,
                                                          const int32_t *vals_in, int32_t n,
                                                          int shift, const int32_t *hist_scan,
                                                          uint32_t *keys_out, int32_t *vals_out) {
    __shared__ int wcount[kWaves][256];
    __shared__ int gbase[256];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) wcount[w][threadIdx.x] = 0;
    gbase[threadIdx.x] = hist_scan[int64_t(threadIdx.x) * gridDim.x + blockIdx.x];
    __syncthreads();

    const int64_t base = int64_t(blockIdx.x) * kSortTile + int64_t(wave) * kWaveItems;
    const uint64_t lanes_below = (uint64_t(1) << lane) - 1;
    uint32_t key[kSortItems];
    int32_t val[kSortItems];
    int rank[kSortItems];
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = base + int64_t(k) * kWaveSize + lane;
        const bool valid = i < n;
        key[k] = valid ? keys_in[i] : 0u;
        val[k] = valid ? vals_in[i] : 0;
        const uint32_t digit = (key[k] >> shift) & 255u;
        uint64_t same = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = (digit >> b) & 1u;
            const uint64_t ones = __ballot(bit);
            same &= bit ? ones : ~ones;
        }
        const int before = __popcll(same & lanes_below);
        const int prior = wcount[wave][digit];
        rank[k] = prior + before;
        __builtin_amdgcn_wave_barrier();
        // the highest lane of each digit group advances the wave's counter
        if (valid && (same >> lane) == 1u) wcount[wave][digit] = prior + __popcll(same);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    {
        int run = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const int c = wcount[w][threadIdx.x];
            wcount[w][threadIdx.x] = run;
            run += c;
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = base + int64_t(k) * kWaveSize + lane;
        if (i < n) {
            const uint32_t digit = (key[k] >> shift) & 255u;
            const int64_t pos = int64_t(gbase[digit]) + wcount[wave][digit] + rank[k];
            keys_out[pos] = key[k];
            vals_out[pos] = val[k];
        }
    }
}

// ---------------------------------------------------------------- interval table

// cell_start[c] = number of kept points with cell < c, for c in [0, n_cells].
// Sorted keys are the kept cells, then n_cells for every dropped point. Slot
// i (0..n) fills the cells in (key[i-1], key[i]] with i; each entry of
// cell_start is written by exactly one slot.
__global__ __launch_bounds__(kBlock) void k_cell_start(const uint32_t *skeys, int32_t n,
                                                       int32_t n_cells, int32_t *cell_start) {
    const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (i > n) return;
    const int64_t prev = (i == 0) ? -1 : int64_t(skeys[i - 1]);
    const int64_t cur = (i == n) ? int64_t(n_cells) : int64_t(skeys[i]);
    for (int64_t c = prev + 1; c <= cur; ++c) cell_start[c] = int32_t(i);
}

__global__ __launch_bounds__(kBlock) void k_cell_stats(const int32_t *cell_start, int32_t n_cells,
                                                       int32_t *stats /* nonempty, max */) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c >= n_cells) return;
    const int32_t cnt = cell_start[c + 1] - cell_start[c];
    if (cnt > 0) {
        atomicAdd(&stats[0], 1);
        atomicMax(&stats[1], cnt);
    }
}

// ---------------------------------------------------------------- work partition
//
// Ray-aligned tiles (see the constants in internal.h). Rows: a point starts
// a new staged row of its tile when the previous depth bin of its pixel is
// dropped or lies in another tile. Every later point of the same run reads
// that row. If a ray leaves a tile and comes back, the pixel is staged twice;
// that wastes one LDS row and changes nothing else.

struct KeyArgs {
    const int32_t *cell_start, *sorted_point;
    int32_t n_cells, HW, W, D, key_cols, key_bins;
    uint32_t *key;            // [n_cells]
    int32_t *nonempty_flag;   // [n_cells + 1]
    int32_t *empty_flag;      // [n_cells + 1]
};

__global__ __launch_bounds__(kBlock) void k_cell_keys(KeyArgs a) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c >= a.n_cells) return;
    const int32_t cnt = a.cell_start[c + 1] - a.cell_start[c];
    a.nonempty_flag[c] = cnt > 0 ? 1 : 0;
    a.empty_flag[c] = cnt > 0 ? 0 : 1;
    if (cnt == 0) return;
    const int32_t p0 = a.sorted_point[a.cell_start[c]];  // the cell's lowest point id
    const int32_t q = p0 / a.HW;                          // n * D + d
    const int32_t n = q / a.D, d = q - n * a.D;
    const int32_t w = p0 % a.W;
    a.key[c] = uint32_t((n * a.key_cols + w / kKeyCols) * a.key_bins + d / kKeyBins);
}

__global__ __launch_bounds__(kBlock) void k_compact_cells(const int32_t *cell_start, int32_t n_cells,
                                                          const uint32_t *key,
                                                          const int32_t *nonempty_pos,
                                                          const int32_t *empty_pos,
                                                          uint32_t *ne_key, int32_t *ne_cell,
                                                          int32_t *empty_cells) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c >= n_cells) return;
    if (cell_start[c + 1] > cell_start[c]) {
        ne_key[nonempty_pos[c]] = key[c];
        ne_cell[nonempty_pos[c]] = c;
    } else {
        empty_cells[empty_pos[c]] = c;
    }
}

// point count of each listed cell, and each cell's position in tile order
__global__ __launch_bounds__(kBlock) void k_listed_counts(const int32_t *listed_cell, int32_t n,
                                                          const int32_t *cell_start,
                                                          int32_t *count_at, int32_t *pos_of_cell) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    const int32_t c = listed_cell[i];
    count_at[i] = cell_start[c + 1] - cell_start[c];
    pos_of_cell[c] = i;
}

__global__ __launch_bounds__(kBlock) void k_group_flags(const uint32_t *key, int32_t n,
                                                        int32_t *flag) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i < n) flag[i] = (i == 0 || key[i] != key[i - 1]) ? 1 : 0;
}

// first listed position of each group (scan = exclusive scan of the flags)
__global__ __launch_bounds__(kBlock) void k_group_first(const int32_t *scan, int32_t n,
                                                        int32_t *group_first) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i > n) return;
    if (i == n) group_first[scan[n]] = n;
    else if (scan[i + 1] != scan[i]) group_first[scan[i]] = i;
}

struct TileFlagArgs {
    const int32_t *group_scan, *group_first, *X;  // X: exclusive scan of the counts
    int32_t n;
    int32_t *flag;
};

__global__ __launch_bounds__(kBlock) void k_tile_flags(TileFlagArgs a) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= a.n) return;
    const int32_t g = a.group_scan[i + 1] - 1;
    const int32_t gf = a.group_first[g];
    const int32_t total = a.X[a.group_first[g + 1]] - a.X[gf];
    constexpr int32_t S = kPointBudget / 2;
    bool start = (i == gf) || ((i - gf) % kMaxTileCells == 0);
    if (!start && total > kPointBudget) {
        const int32_t here = a.X[i] - a.X[gf], prev = a.X[i - 1] - a.X[gf];
        const int32_t n_here = a.X[i + 1] - a.X[i], n_prev = a.X[i] - a.X[i - 1];
        start = (here / S != prev / S) || n_here > S || n_prev > S;
    }
    a.flag[i] = start ? 1 : 0;
}

// tile_cell_begin[t] = first listed position of tile t; tile_of_cell per cell
__global__ __launch_bounds__(kBlock) void k_tile_emit(const int32_t *tile_scan, int32_t n,
                                                      const int32_t *listed_cell,
                                                      int32_t *tile_cell_begin,
                                                      int32_t *tile_of_cell) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i > n) return;
    if (i == n) {
        tile_cell_begin[tile_scan[n]] = n;
        return;
    }
    if (tile_scan[i + 1] != tile_scan[i]) tile_cell_begin[tile_scan[i]] = i;
    tile_of_cell[listed_cell[i]] = tile_scan[i + 1] - 1;
}

// Points in tile order: a cell's run of the canonical order moves as a block.
__global__ __launch_bounds__(kBlock) void k_comp_points(const int32_t *sorted_point, int32_t n_kept,
                                                        const int32_t *cell_of_point,
                                                        const int32_t *cell_start,
                                                        const int32_t *pos_of_cell,
                                                        const int32_t *comp_cell_start,
                                                        int32_t *comp_point, int32_t *pos_of_point) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n_kept) return;
    const int32_t p = sorted_point[i];
    const int32_t c = cell_of_point[p];
    const int32_t ci = comp_cell_start[pos_of_cell[c]] + (i - cell_start[c]);
    comp_point[ci] = p;
    pos_of_point[p] = ci;
}

// 1 where a point starts a run of its pixel inside its tile
__global__ __launch_bounds__(kBlock) void k_run_flags(const int32_t *comp_point, int32_t n_kept,
                                                      const int32_t *cell_of_point,
                                                      const int32_t *tile_of_cell, int32_t HW,
                                                      FastDiv div_hw, FastDiv div_d, int32_t D,
                                                      int32_t *flag) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n_kept) return;
    const int32_t p = comp_point[i];
    const uint32_t q = fdiv(uint32_t(p), div_hw);
    const int32_t d = int32_t(q) - int32_t(fdiv(q, div_d)) * D;
    const int32_t prev = d > 0 ? cell_of_point[p - HW] : -1;
    flag[i] = (prev < 0 || tile_of_cell[prev] != tile_of_cell[cell_of_point[p]]) ? 1 : 0;
}

__global__ __launch_bounds__(kBlock) void k_tile_row_begin(const int32_t *tile_cell_begin,
                                                           const int32_t *comp_cell_start,
                                                           const int32_t *row_scan, int32_t n_tiles,
                                                           int32_t *tile_row_begin) {
    const int32_t t = blockIdx.x * kBlock + threadIdx.x;
    if (t <= n_tiles) tile_row_begin[t] = row_scan[comp_cell_start[tile_cell_begin[t]]];
}

// One thread per pixel walks its depth bins in order, names the staged row
// of each run and gives every point its row relative to its tile.
__global__ __launch_bounds__(kBlock) void k_rows(const int32_t *cell_of_point,
                                                 const int32_t *pos_of_point,
                                                 const int32_t *tile_of_cell,
                                                 const int32_t *row_scan,
                                                 const int32_t *tile_row_begin, int32_t n_pix,
                                                 int32_t HW, int32_t D, int32_t *row_pix,
                                                 int32_t *comp_row) {
    const int32_t pixel = blockIdx.x * kBlock + threadIdx.x;
    if (pixel >= n_pix) return;
    const int32_t n = pixel / HW, hw = pixel - n * HW;
    int32_t row = 0;
    for (int32_t d = 0; d < D; ++d) {
        const int32_t p = (n * D + d) * HW + hw;
        const int32_t c = cell_of_point[p];
        if (c < 0) continue;
        const int32_t i = pos_of_point[p];
        if (row_scan[i + 1] != row_scan[i]) {
            row = row_scan[i];
            row_pix[row] = pixel;
        }
        comp_row[i] = row - tile_row_begin[tile_of_cell[c]];
    }
}

// Per-tile header, heavy flag and cost (for splitting tiles over the
// persistent workgroups): points, plus rows and cells, which also cost time.
__global__ __launch_bounds__(kBlock) void k_tile_headers(const int32_t *tile_cell_begin,
                                                         const int32_t *tile_row_begin,
                                                         const int32_t *comp_cell_start,
                                                         int32_t n_tiles, int32_t *hdr,
                                                         int32_t *heavy_flag, int32_t *cost) {
    const int32_t t = blockIdx.x * kBlock + threadIdx.x;
    if (t >= n_tiles) return;
    const int32_t tcb = tile_cell_begin[t], ncell = tile_cell_begin[t + 1] - tcb;
    const int32_t tpb = comp_cell_start[tcb], npts = comp_cell_start[tcb + ncell] - tpb;
    const int32_t trb = tile_row_begin[t], nrows = tile_row_begin[t + 1] - trb;
    int32_t *h = hdr + 8 * int64_t(t);
    h[0] = tcb;
    h[1] = ncell;
    h[2] = tpb;
    h[3] = npts;
    h[4] = trb;
    h[5] = nrows;
    h[6] = 0;
    h[7] = 0;
    const bool heavy = npts > kPointBudget;
    heavy_flag[t] = heavy ? 1 : 0;
    cost[t] = heavy ? 0 : npts + 2 * nrows + 4 * ncell + 64;
}

__global__ __launch_bounds__(kBlock) void k_heavy_list(const int32_t *heavy_scan, int32_t n_tiles,
                                                       int32_t *heavy_tiles) {
    const int32_t t = blockIdx.x * kBlock + threadIdx.x;
    if (t < n_tiles && heavy_scan[t + 1] != heavy_scan[t]) heavy_tiles[heavy_scan[t]] = t;
}

// group_tile_begin[w] = first tile whose running cost reaches w/G of the total
__global__ __launch_bounds__(kBlock) void k_group_ranges(const int32_t *cost_scan, int32_t n_tiles,
                                                         int32_t *group_tile_begin) {
    const int32_t w = blockIdx.x * kBlock + threadIdx.x;
    if (w > kPersistentGroups) return;
    const int64_t total = cost_scan[n_tiles];
    const int64_t target = total * w / kPersistentGroups;
    int32_t lo = 0, hi = n_tiles;  // first t with cost_scan[t] >= target
    while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (cost_scan[mid] < target) lo = mid + 1;
        else hi = mid;
    }
    group_tile_begin[w] = (w == kPersistentGroups) ? n_tiles : lo;
}

int blocks_for(int64_t n) { return int((n + kBlock - 1) / kBlock); }

template <typename T>
int dev_alloc(T **p, size_t count, const char *what) {
    *p = nullptr;
    hipError_t e = hipMalloc(reinterpret_cast<void **>(p), (count ? count : 1) * sizeof(T));
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) {
        (void)hipGetLastError();
        return bevpool_fail(BEVPOOL_ERR_OOM, "out of device memory allocating %s (%zu bytes)", what,
                            count * sizeof(T));
    }
    if (e != hipSuccess) return bevpool_hip_fail(e, what);
    return BEVPOOL_OK;
}

// Exclusive scan of data[0..n] in place; data[n] must be 0 on entry and
// holds the total afterwards.
void scan_with_total(int32_t *data, int64_t n, int32_t *scratch_total, hipStream_t stream) {
    hipLaunchKernelGGL(k_scan, dim3(1), dim3(kScanBlock), 0, stream, data, n + 1, scratch_total);
}

}  // namespace
}  // namespace bevpool

using namespace bevpool;

int bevpool_build_plan(const double *intrinsics, const double *extrinsics,
                       const bevpool_geometry &g, hipStream_t stream, bevpool_plan_s *plan) {
    const int64_t np64 = int64_t(g.n_cams) * g.n_depth * g.feat_h * g.feat_w;
    const int32_t np = int32_t(np64);
    const int32_t n_cells = g.nx * g.ny;
    const int32_t HW = g.feat_h * g.feat_w;
    const int32_t n_pix = g.n_cams * HW;
    plan->n_points = np64;
    plan->n_cells = n_cells;

    int rc;
    if ((rc = dev_alloc(&plan->cell_of_point, size_t(np), "cell_of_point"))) return rc;
    if ((rc = dev_alloc(&plan->sorted_point, size_t(np), "sorted_point"))) return rc;
    if ((rc = dev_alloc(&plan->cell_start, size_t(n_cells) + 1, "cell_start"))) return rc;

    // temporaries, freed on every exit path below
    const int64_t sort_cap = np64 > n_cells ? np64 : int64_t(n_cells);
    const int sort_tiles_cap = int((sort_cap + kSortTile - 1) / kSortTile);
    double *d_calib = nullptr;
    uint32_t *keys_a = nullptr, *keys_b = nullptr, *cell_key = nullptr;
    int32_t *vals_b = nullptr, *hist = nullptr, *small = nullptr;
    int32_t *flag_a = nullptr, *flag_b = nullptr, *group_first = nullptr;
    int32_t *tile_of_cell = nullptr, *pos_of_cell = nullptr, *pos_of_point = nullptr;
    int32_t *row_scan = nullptr;
    auto cleanup = [&]() {
        (void)hipFree(d_calib);
        (void)hipFree(keys_a);
        (void)hipFree(keys_b);
        (void)hipFree(cell_key);
        (void)hipFree(vals_b);
        (void)hipFree(hist);
        (void)hipFree(small);
        (void)hipFree(flag_a);
        (void)hipFree(flag_b);
        (void)hipFree(group_first);
        (void)hipFree(tile_of_cell);
        (void)hipFree(pos_of_cell);
        (void)hipFree(pos_of_point);
        (void)hipFree(row_scan);
    };
    auto launch_ok = [](int64_t n) { return n > 0; };

    // stable LSD radix sort of (keys, vals)[0, n) on the low `bits` bits; the
    // result ends in (keys, vals)
    auto radix_sort = [&](uint32_t *keys, int32_t *vals, int32_t n, int bits) -> int {
        if (n <= 0) return BEVPOOL_OK;
        const int tiles = int((int64_t(n) + kSortTile - 1) / kSortTile);
        const int passes = (bits + 7) / 8;
        uint32_t *kin = keys, *kout = keys == keys_a ? keys_b : keys_a;
        int32_t *vin = vals, *vout = vals_b;
        for (int pass = 0; pass < passes; ++pass) {
            const int shift = 8 * pass;
            hipLaunchKernelGGL(k_radix_hist, dim3(tiles), dim3(kBlock), 0, stream, kin, n, shift, hist);
            hipLaunchKernelGGL(k_scan, dim3(1), dim3(kScanBlock), 0, stream, hist,
                               int64_t(tiles) * 256, small + 3);
            hipLaunchKernelGGL(k_radix_scatter, dim3(tiles), dim3(kBlock), 0, stream, kin, vin, n,
                               shift, hist, kout, vout);
            BEVPOOL_HIP(hipGetLastError());
            std::swap(kin, kout);
            std::swap(vin, vout);
        }
        if (kin != keys)
            BEVPOOL_HIP(hipMemcpyAsync(keys, kin, sizeof(uint32_t) * size_t(n),
                                       hipMemcpyDeviceToDevice, stream));
        if (vin != vals)
            BEVPOOL_HIP(hipMemcpyAsync(vals, vin, sizeof(int32_t) * size_t(n),
                                       hipMemcpyDeviceToDevice, stream));
        return BEVPOOL_OK;
    };
    auto bits_for = [](int64_t max_key) {
        int b = 1;
        while ((int64_t(1) << b) <= max_key) ++b;
        return b;
    };

    auto run = [&]() -> int {
        int rc2;
        if ((rc2 = dev_alloc(&d_calib, size_t(g.n_cams) * 16, "calibration"))) return rc2;
        if ((rc2 = dev_alloc(&keys_a, size_t(sort_cap), "sort keys"))) return rc2;
        if ((rc2 = dev_alloc(&keys_b, size_t(sort_cap), "sort keys"))) return rc2;
        if ((rc2 = dev_alloc(&vals_b, size_t(sort_cap), "sort values"))) return rc2;
        if ((rc2 = dev_alloc(&cell_key, size_t(n_cells), "cell keys"))) return rc2;
        if ((rc2 = dev_alloc(&hist, size_t(sort_tiles_cap) * 256, "radix histogram"))) return rc2;
        if ((rc2 = dev_alloc(&small, 4, "plan counters"))) return rc2;
        if ((rc2 = dev_alloc(&flag_a, size_t(n_cells) + 1, "flags"))) return rc2;
        if ((rc2 = dev_alloc(&flag_b, size_t(n_cells) + 1, "flags"))) return rc2;
        if ((rc2 = dev_alloc(&group_first, size_t(n_cells) + 1, "group starts"))) return rc2;
        if ((rc2 = dev_alloc(&tile_of_cell, size_t(n_cells), "tile of cell"))) return rc2;
        if ((rc2 = dev_alloc(&pos_of_cell, size_t(n_cells), "cell positions"))) return rc2;
        if ((rc2 = dev_alloc(&pos_of_point, size_t(np), "point positions"))) return rc2;

        BEVPOOL_HIP(hipMemcpyAsync(d_calib, intrinsics, sizeof(double) * 4 * g.n_cams,
                                   hipMemcpyHostToDevice, stream));
        BEVPOOL_HIP(hipMemcpyAsync(d_calib + 4 * g.n_cams, extrinsics,
                                   sizeof(double) * 12 * g.n_cams, hipMemcpyHostToDevice, stream));
        BEVPOOL_HIP(hipMemsetAsync(small, 0, 4 * sizeof(int32_t), stream));

        ProjectArgs pa;
        pa.intr = d_calib;
        pa.extr = d_calib + 4 * g.n_cams;
        pa.g = g;
        pa.div_w = make_fastdiv(uint32_t(g.feat_w));
        pa.div_h = make_fastdiv(uint32_t(g.feat_h));
        pa.div_d = make_fastdiv(uint32_t(g.n_depth));
        pa.n_points = np;
        pa.n_cells = n_cells;
        pa.cell_of_point = plan->cell_of_point;
        pa.keys = keys_a;
        pa.vals = plan->sorted_point;
        hipLaunchKernelGGL(k_project, dim3(blocks_for(np)), dim3(kBlock), 0, stream, pa);
        BEVPOOL_HIP(hipGetLastError());

        // canonical order: points by (cell, id); dropped points last
        if ((rc2 = radix_sort(keys_a, plan->sorted_point, np, bits_for(n_cells)))) return rc2;
        hipLaunchKernelGGL(k_cell_start, dim3(blocks_for(int64_t(np) + 1)), dim3(kBlock), 0,
                           stream, keys_a, np, n_cells, plan->cell_start);
        hipLaunchKernelGGL(k_cell_stats, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, small);

        // cells with points, keyed along the rays; cells without points listed
        const int32_t key_cols = (g.feat_w + kKeyCols - 1) / kKeyCols;
        const int32_t key_bins = (g.n_depth + kKeyBins - 1) / kKeyBins;
        KeyArgs ka;
        ka.cell_start = plan->cell_start;
        ka.sorted_point = plan->sorted_point;
        ka.n_cells = n_cells;
        ka.HW = HW;
        ka.W = g.feat_w;
        ka.D = g.n_depth;
        ka.key_cols = key_cols;
        ka.key_bins = key_bins;
        ka.key = cell_key;
        ka.nonempty_flag = flag_a;
        ka.empty_flag = flag_b;
        BEVPOOL_HIP(hipMemsetAsync(flag_a, 0, sizeof(int32_t) * (size_t(n_cells) + 1), stream));
        BEVPOOL_HIP(hipMemsetAsync(flag_b, 0, sizeof(int32_t) * (size_t(n_cells) + 1), stream));
        hipLaunchKernelGGL(k_cell_keys, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream, ka);
        scan_with_total(flag_a, n_cells, small + 3, stream);
        scan_with_total(flag_b, n_cells, small + 3, stream);
        BEVPOOL_HIP(hipGetLastError());
        int32_t host[2], counts2[2];
        BEVPOOL_HIP(hipMemcpyAsync(host, small, sizeof(host), hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipMemcpyAsync(&counts2[0], flag_a + n_cells, sizeof(int32_t),
                                   hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipMemcpyAsync(&counts2[1], flag_b + n_cells, sizeof(int32_t),
                                   hipMemcpyDeviceToHost, stream));
        int32_t kept;
        BEVPOOL_HIP(hipMemcpyAsync(&kept, plan->cell_start + n_cells, sizeof(kept),
                                   hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        plan->n_nonempty = host[0];
        plan->max_per_cell = host[1];
        plan->n_kept = kept;
        const int32_t n_ne = counts2[0];
        plan->n_empty = counts2[1];

        if ((rc2 = dev_alloc(&plan->tile_cells, size_t(n_ne), "tile_cells"))) return rc2;
        if ((rc2 = dev_alloc(&plan->comp_cell_start, size_t(n_ne) + 1, "comp_cell_start"))) return rc2;
        if ((rc2 = dev_alloc(&plan->empty_cells, size_t(plan->n_empty), "empty_cells"))) return rc2;
        // compact into (key, cell) pairs in keys_b / vals_b's partner buffers
        uint32_t *ne_key = keys_a;     // free again after k_cell_start
        int32_t *ne_cell = plan->tile_cells;
        hipLaunchKernelGGL(k_compact_cells, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, cell_key, flag_a, flag_b, ne_key, ne_cell,
                           plan->empty_cells);
        BEVPOOL_HIP(hipGetLastError());
        const int64_t max_key = int64_t(g.n_cams) * key_cols * key_bins;
        if ((rc2 = radix_sort(ne_key, ne_cell, n_ne, bits_for(max_key)))) return rc2;

        // point counts in tile order and their running sum
        BEVPOOL_HIP(hipMemsetAsync(plan->comp_cell_start, 0, sizeof(int32_t) * (size_t(n_ne) + 1),
                                   stream));
        if (launch_ok(n_ne)) {
            hipLaunchKernelGGL(k_listed_counts, dim3(blocks_for(n_ne)), dim3(kBlock), 0, stream,
                               plan->tile_cells, n_ne, plan->cell_start, plan->comp_cell_start,
                               pos_of_cell);
        }
        scan_with_total(plan->comp_cell_start, n_ne, small + 3, stream);

        // key groups, then tiles
        BEVPOOL_HIP(hipMemsetAsync(flag_a, 0, sizeof(int32_t) * (size_t(n_ne) + 1), stream));
        BEVPOOL_HIP(hipMemsetAsync(flag_b, 0, sizeof(int32_t) * (size_t(n_ne) + 1), stream));
        if (launch_ok(n_ne))
            hipLaunchKernelGGL(k_group_flags, dim3(blocks_for(n_ne)), dim3(kBlock), 0, stream,
                               ne_key, n_ne, flag_a);
        scan_with_total(flag_a, n_ne, small + 3, stream);
        hipLaunchKernelGGL(k_group_first, dim3(blocks_for(int64_t(n_ne) + 1)), dim3(kBlock), 0,
                           stream, flag_a, n_ne, group_first);
        TileFlagArgs ta;
        ta.group_scan = flag_a;
        ta.group_first = group_first;
        ta.X = plan->comp_cell_start;
        ta.n = n_ne;
        ta.flag = flag_b;
        if (launch_ok(n_ne))
            hipLaunchKernelGGL(k_tile_flags, dim3(blocks_for(n_ne)), dim3(kBlock), 0, stream, ta);
        scan_with_total(flag_b, n_ne, small + 3, stream);
        BEVPOOL_HIP(hipGetLastError());
        BEVPOOL_HIP(hipMemcpyAsync(&plan->n_tiles, flag_b + n_ne, sizeof(int32_t),
                                   hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        const int32_t n_tiles = plan->n_tiles;
        if ((rc2 = dev_alloc(&plan->tile_cell_begin, size_t(n_tiles) + 1, "tile_cell_begin"))) return rc2;
        if ((rc2 = dev_alloc(&plan->tile_row_begin, size_t(n_tiles) + 1, "tile_row_begin"))) return rc2;
        hipLaunchKernelGGL(k_tile_emit, dim3(blocks_for(int64_t(n_ne) + 1)), dim3(kBlock), 0,
                           stream, flag_b, n_ne, plan->tile_cells, plan->tile_cell_begin,
                           tile_of_cell);
        BEVPOOL_HIP(hipGetLastError());

        // points in tile order, staged rows and each point's row
        if ((rc2 = dev_alloc(&plan->comp_point, size_t(kept), "comp_point"))) return rc2;
        if ((rc2 = dev_alloc(&plan->comp_row, size_t(kept), "comp_row"))) return rc2;
        if ((rc2 = dev_alloc(&row_scan, size_t(kept) + 1, "row scan"))) return rc2;
        BEVPOOL_HIP(hipMemsetAsync(row_scan, 0, sizeof(int32_t) * (size_t(kept) + 1), stream));
        if (launch_ok(kept)) {
            hipLaunchKernelGGL(k_comp_points, dim3(blocks_for(kept)), dim3(kBlock), 0, stream,
                               plan->sorted_point, kept, plan->cell_of_point, plan->cell_start,
                               pos_of_cell, plan->comp_cell_start, plan->comp_point, pos_of_point);
            hipLaunchKernelGGL(k_run_flags, dim3(blocks_for(kept)), dim3(kBlock), 0, stream,
                               plan->comp_point, kept, plan->cell_of_point, tile_of_cell, HW,
                               make_fastdiv(uint32_t(HW)), make_fastdiv(uint32_t(g.n_depth)),
                               g.n_depth, row_scan);
        }
        scan_with_total(row_scan, kept, small + 3, stream);
        hipLaunchKernelGGL(k_tile_row_begin, dim3(blocks_for(int64_t(n_tiles) + 1)), dim3(kBlock), 0,
                           stream, plan->tile_cell_begin, plan->comp_cell_start, row_scan, n_tiles,
                           plan->tile_row_begin);
        BEVPOOL_HIP(hipGetLastError());
        int32_t n_rows;
        BEVPOOL_HIP(hipMemcpyAsync(&n_rows, row_scan + kept, sizeof(n_rows), hipMemcpyDeviceToHost,
                                   stream));
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        plan->n_rows = n_rows;
        if ((rc2 = dev_alloc(&plan->row_pix, size_t(n_rows), "row_pix"))) return rc2;
        hipLaunchKernelGGL(k_rows, dim3(blocks_for(n_pix)), dim3(kBlock), 0, stream,
                           plan->cell_of_point, pos_of_point, tile_of_cell, row_scan,
                           plan->tile_row_begin, n_pix, HW, g.n_depth, plan->row_pix,
                           plan->comp_row);
        BEVPOOL_HIP(hipGetLastError());

        // headers, heavy tiles and the persistent workgroups' tile runs
        if ((rc2 = dev_alloc(&plan->tile_hdr, size_t(n_tiles) * 8, "tile_hdr"))) return rc2;
        if ((rc2 = dev_alloc(&plan->group_tile_begin, size_t(kPersistentGroups) + 1, "tile runs"))) return rc2;
        BEVPOOL_HIP(hipMemsetAsync(flag_a, 0, sizeof(int32_t) * (size_t(n_tiles) + 1), stream));
        BEVPOOL_HIP(hipMemsetAsync(flag_b, 0, sizeof(int32_t) * (size_t(n_tiles) + 1), stream));
        if (launch_ok(n_tiles))
            hipLaunchKernelGGL(k_tile_headers, dim3(blocks_for(n_tiles)), dim3(kBlock), 0, stream,
                               plan->tile_cell_begin, plan->tile_row_begin, plan->comp_cell_start,
                               n_tiles, plan->tile_hdr, flag_a, flag_b);
        scan_with_total(flag_a, n_tiles, small + 3, stream);
        scan_with_total(flag_b, n_tiles, small + 3, stream);
        hipLaunchKernelGGL(k_group_ranges, dim3(blocks_for(kPersistentGroups + 1)), dim3(kBlock), 0,
                           stream, flag_b, n_tiles, plan->group_tile_begin);
        BEVPOOL_HIP(hipMemcpyAsync(&plan->n_heavy, flag_a + n_tiles, sizeof(int32_t),
                                   hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        if ((rc2 = dev_alloc(&plan->heavy_tiles, size_t(plan->n_heavy), "heavy_tiles"))) return rc2;
        if (launch_ok(n_tiles))
            hipLaunchKernelGGL(k_heavy_list, dim3(blocks_for(n_tiles)), dim3(kBlock), 0, stream,
                               flag_a, n_tiles, plan->heavy_tiles);
        BEVPOOL_HIP(hipGetLastError());
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        return BEVPOOL_OK;
    };
    rc = run();
    if (rc != BEVPOOL_OK) (void)hipStreamSynchronize(stream);
    cleanup();
    return rc;
}
