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
//   k_tile_flags / k_scan / k_tile_emit   work partition of the forward pass
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

__device__ __forceinline__ bool tile_starts_at(const int32_t *cs, int32_t c) {
    if (c == 0) return true;
    const int64_t here = int64_t(kCellWeight) * c + cs[c];
    const int64_t prev = int64_t(kCellWeight) * (c - 1) + cs[c - 1];
    const int32_t n_here = cs[c + 1] - cs[c];
    const int32_t n_prev = cs[c] - cs[c - 1];
    return (here / kTilePath != prev / kTilePath) || n_here > kHeavyPoints || n_prev > kHeavyPoints;
}

__global__ __launch_bounds__(kBlock) void k_tile_flags(const int32_t *cs, int32_t n_cells,
                                                       int32_t *flags) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c < n_cells) flags[c] = tile_starts_at(cs, c) ? 1 : 0;
}

__global__ __launch_bounds__(kBlock) void k_tile_emit(const int32_t *cs, int32_t n_cells,
                                                      const int32_t *slot, const int32_t *n_tiles,
                                                      int32_t *tile_cell) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c < n_cells && tile_starts_at(cs, c)) tile_cell[slot[c]] = c;
    if (c == 0) tile_cell[*n_tiles] = n_cells;
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

}  // namespace
}  // namespace bevpool

using namespace bevpool;

int bevpool_build_plan(const double *intrinsics, const double *extrinsics,
                       const bevpool_geometry &g, hipStream_t stream, bevpool_plan_s *plan) {
    const int64_t np64 = int64_t(g.n_cams) * g.n_depth * g.feat_h * g.feat_w;
    const int32_t np = int32_t(np64);
    const int32_t n_cells = g.nx * g.ny;
    plan->n_points = np64;
    plan->n_cells = n_cells;

    int rc;
    if ((rc = dev_alloc(&plan->cell_of_point, size_t(np), "cell_of_point"))) return rc;
    if ((rc = dev_alloc(&plan->sorted_point, size_t(np), "sorted_point"))) return rc;
    if ((rc = dev_alloc(&plan->cell_start, size_t(n_cells) + 1, "cell_start"))) return rc;
    if ((rc = dev_alloc(&plan->tile_cell, size_t(n_cells) + 1, "tile_cell"))) return rc;

    // temporaries, freed on every exit path below
    const int sort_tiles = int((np64 + kSortTile - 1) / kSortTile);
    int bits = 1;
    while ((int64_t(1) << bits) <= int64_t(n_cells)) ++bits;  // keys are 0..n_cells
    const int passes = (bits + 7) / 8;
    double *d_calib = nullptr;
    uint32_t *keys_a = nullptr, *keys_b = nullptr;
    int32_t *vals_b = nullptr, *hist = nullptr, *small = nullptr, *flags = nullptr;
    auto cleanup = [&]() {
        (void)hipFree(d_calib);
        (void)hipFree(keys_a);
        (void)hipFree(keys_b);
        (void)hipFree(vals_b);
        (void)hipFree(hist);
        (void)hipFree(small);
        (void)hipFree(flags);
    };
    auto run = [&]() -> int {
        int rc2;
        if ((rc2 = dev_alloc(&d_calib, size_t(g.n_cams) * 16, "calibration"))) return rc2;
        if ((rc2 = dev_alloc(&keys_a, size_t(np), "sort keys"))) return rc2;
        if ((rc2 = dev_alloc(&keys_b, size_t(np), "sort keys"))) return rc2;
        if ((rc2 = dev_alloc(&vals_b, size_t(np), "sort values"))) return rc2;
        if ((rc2 = dev_alloc(&hist, size_t(sort_tiles) * 256, "radix histogram"))) return rc2;
        if ((rc2 = dev_alloc(&small, 4, "plan counters"))) return rc2;
        if ((rc2 = dev_alloc(&flags, size_t(n_cells) + 1, "tile flags"))) return rc2;

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

        // LSD radix sort; buffers alternate so the last pass lands in
        // plan->sorted_point (values) whatever the number of passes
        uint32_t *kin = keys_a, *kout = keys_b;
        int32_t *vin = plan->sorted_point, *vout = vals_b;
        for (int pass = 0; pass < passes; ++pass) {
            const int shift = 8 * pass;
            hipLaunchKernelGGL(k_radix_hist, dim3(sort_tiles), dim3(kBlock), 0, stream, kin, np,
                               shift, hist);
            hipLaunchKernelGGL(k_scan, dim3(1), dim3(kScanBlock), 0, stream, hist,
                               int64_t(sort_tiles) * 256, small + 3);
            hipLaunchKernelGGL(k_radix_scatter, dim3(sort_tiles), dim3(kBlock), 0, stream, kin,
                               vin, np, shift, hist, kout, vout);
            BEVPOOL_HIP(hipGetLastError());
            std::swap(kin, kout);
            std::swap(vin, vout);
        }
        if (vin != plan->sorted_point)
            BEVPOOL_HIP(hipMemcpyAsync(plan->sorted_point, vin, sizeof(int32_t) * size_t(np),
                                       hipMemcpyDeviceToDevice, stream));

        hipLaunchKernelGGL(k_cell_start, dim3(blocks_for(int64_t(np) + 1)), dim3(kBlock), 0,
                           stream, kin, np, n_cells, plan->cell_start);
        hipLaunchKernelGGL(k_cell_stats, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, small);
        hipLaunchKernelGGL(k_tile_flags, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, flags);
        hipLaunchKernelGGL(k_scan, dim3(1), dim3(kScanBlock), 0, stream, flags, int64_t(n_cells),
                           small + 2);
        hipLaunchKernelGGL(k_tile_emit, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, flags, small + 2, plan->tile_cell);
        BEVPOOL_HIP(hipGetLastError());

        int32_t stats[4];
        int32_t kept;
        BEVPOOL_HIP(hipMemcpyAsync(stats, small, sizeof(stats), hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipMemcpyAsync(&kept, plan->cell_start + n_cells, sizeof(kept),
                                   hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        plan->n_nonempty = stats[0];
        plan->max_per_cell = stats[1];
        plan->n_tiles = stats[2];
        plan->n_kept = kept;
        return BEVPOOL_OK;
    };
    rc = run();
    if (rc != BEVPOOL_OK) (void)hipStreamSynchronize(stream);
    cleanup();
    return rc;
}
