// Plan building for BEV pooling: the camera-fixed point-to-cell association
// (BEVFusion, arXiv 2205.13542, Sec. III-B, "Precomputation" paragraph:
// compute each frustum point's 3-D coordinate and grid index once, sort the
// points by grid index and record their ranks).
//
// Kernels, in launch order:
//   k_project      one thread per point: camera ray -> ego frame -> cell id
//   k_radix_hist   } stable LSD radix sort of (cell, point id), digits of
//                  } at most 9 bits;
//   k_scan...      } input in id order, so ties stay in id order (scans:
//   k_radix_scatter} one workgroup for a short array, else chunk sums,
//                    their scan and per-chunk scans from the offsets)
//   k_cell_start   interval table from the sorted keys
//   k_cell_stats   non-empty cells and the largest interval
//   k_combo_walk ... k_generic_runs   work partition of the forward pass:
//                  clean combos, the column table, empty cells, the
//                  partial-sum slots of multi-combo cells, generic cells and
//                  their runs
//
// The geometry is evaluated in IEEE double with the file built without
// floating-point contraction, in one fixed expression order, so the cell ids
// equal those of any plain CPU evaluation of the same expressions.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <utility>

#include "internal.h"

#pragma clang fp contract(off)

namespace bevpool {
namespace {

constexpr int kSortItems = 8;                       // keys per thread per tile
constexpr int kSortTile = kBlock * kSortItems;      // 2048 keys per workgroup
constexpr int kWaveItems = kWaveSize * kSortItems;  // 512 keys per wave
constexpr int kRadixBits = 9;                       // digit bits per pass, at most
constexpr int kRadixBins = 1 << kRadixBits;         // 512 digits, at most two per thread

// A sort on `bits` key bits takes the fewest passes of at most kRadixBits
// bits, with the bits split evenly over them (17-bit cell ids: two passes of
// 9; 19 bits: three of 7, whose 128-digit histograms are cheaper than 512).
constexpr int radix_passes(int bits) { return (bits + kRadixBits - 1) / kRadixBits; }
constexpr int radix_digit_bits(int bits) {
    return (bits + radix_passes(bits) - 1) / radix_passes(bits);
}
constexpr int kScanBlock = 1024;
constexpr int kScanItems = 4;
constexpr int kScanChunk = kScanBlock * kScanItems;  // elements per workgroup of a multi-block scan
constexpr int kScanOneBlockChunks = 8;               // scans of up to 8 chunks take one workgroup
static_assert(kBlock == 256, "a sort tile is four waves of 512 keys");

constexpr int kArgCams = 16;   // cameras whose calibration travels in the kernel arguments

struct ProjectArgs {
    const double *intr;  // [N][4] in device memory, or null: the calibration is in cal
    const double *extr;  // [N][12]
    double cal[kArgCams * 16];   // [N][4] intrinsics, then [N][12] extrinsics (intr null)
    bevpool_geometry g;
    FastDiv div_w, div_h, div_d;
    int32_t n_points, n_cells, nz;
    int32_t *cell_of_point;
    uint32_t *keys;
    int32_t *vals;
};

// Sec. III-B, first paragraph: the pixel's ray at depth bin d, in the ego
// frame, quantised at the cell size, z like x and y; points outside the grid
// or the nz stacked z slabs are dropped. Cell id (iy * nx + ix) * nz + iz.
// Sort key = cell id, or n_cells for a dropped point (last).
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

    const double *I = a.intr ? a.intr + 4 * n : a.cal + 4 * n;
    const double *E = a.intr ? a.extr + 12 * n : a.cal + 4 * g.n_cams + 12 * n;
    const double fx = I[0], fy = I[1], cx = I[2], cy = I[3];
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
    if (qx >= 0.0 && qx < double(g.nx) && qy >= 0.0 && qy < double(g.ny) && qz >= 0.0 &&
        qz < double(a.nz))
        cell = (int32_t(qy) * g.nx + int32_t(qx)) * a.nz + int32_t(qz);
    a.cell_of_point[p] = cell;
    a.keys[p] = cell >= 0 ? uint32_t(cell) : uint32_t(a.n_cells);
    a.vals[p] = p;
}

// A stored association (bevpool_plan_import): the sort keys and point ids
// from a cell map validated on the host.
__global__ __launch_bounds__(kBlock) void k_keys_from_cells(const int32_t *cell_of_point,
                                                            int32_t n_points, int32_t n_cells,
                                                            uint32_t *keys, int32_t *vals) {
    const int32_t p = blockIdx.x * kBlock + threadIdx.x;
    if (p >= n_points) return;
    const int32_t cell = cell_of_point[p];
    keys[p] = cell >= 0 ? uint32_t(cell) : uint32_t(n_cells);
    vals[p] = p;
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

// Multi-block exclusive scan, for arrays longer than one chunk: each
// workgroup sums its chunk, one workgroup scans the chunk sums (k_scan),
// and each workgroup scans its chunk again from its offset.
__global__ __launch_bounds__(kScanBlock) void k_scan_sums(const int32_t *data, int64_t n,
                                                          int32_t *sums) {
    __shared__ int lds[kScanBlock / kWaveSize];
    const int64_t i0 = int64_t(blockIdx.x) * kScanChunk + int64_t(threadIdx.x) * kScanItems;
    int local = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) local += (i0 + k < n) ? data[i0 + k] : 0;
    int total;
    (void)block_exclusive_scan<kScanBlock>(local, lds, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kScanBlock) void k_scan_apply(int32_t *data, int64_t n,
                                                           const int32_t *offsets) {
    __shared__ int lds[kScanBlock / kWaveSize];
    const int64_t i0 = int64_t(blockIdx.x) * kScanChunk + int64_t(threadIdx.x) * kScanItems;
    int v[kScanItems];
    int local = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = (i0 + k < n) ? data[i0 + k] : 0;
        local += v[k];
    }
    int total;
    int run = offsets[blockIdx.x] + block_exclusive_scan<kScanBlock>(local, lds, &total);
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        if (i0 + k < n) data[i0 + k] = run;
        run += v[k];
    }
}

// ---------------------------------------------------------------- radix sort

// Digit histogram of each 2048-key tile, stored digit-major:
// hist[digit * n_tiles + tile], so an exclusive scan of the whole array
// gives every (digit, tile) its first output slot in stable order.
// Digit counts of one tile: hist[digit * tiles + tile], digits of dbits
// bits (dbits <= kRadixBits) from bit `shift` on.
__global__ __launch_bounds__(kBlock) void k_radix_hist(const uint32_t *keys, int32_t n,
                                                       int shift, int dbits, int32_t *hist) {
    __shared__ int cnt[kRadixBins];
    const int bins = 1 << dbits;
    const uint32_t mask = uint32_t(bins) - 1u;
    for (int d = threadIdx.x; d < bins; d += kBlock) cnt[d] = 0;
    __syncthreads();
    const int64_t base = int64_t(blockIdx.x) * kSortTile;
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = base + int64_t(k) * kBlock + threadIdx.x;
        if (i < n) atomicAdd(&cnt[(keys[i] >> shift) & mask], 1);
    }
    __syncthreads();
    for (int d = threadIdx.x; d < bins; d += kBlock)
        hist[int64_t(d) * gridDim.x + blockIdx.x] = cnt[d];
}

// Stable scatter. Wave w of a tile owns keys [w*512, (w+1)*512) of the tile
// and walks them 64 at a time in order. Within a step, a key's rank among
// equal digits comes from one ballot per digit bit: lanes whose ballots
// agree on every bit hold the same digit. A per-wave LDS counter per
// digit carries ranks across steps. Per-wave counts are then prefixed across
// the waves and added to the scanned global offsets.
__global__ __launch_bounds__(kBlock) void k_radix_scatter(const uint32_t *keys_in,
                                                          const int32_t *vals_in, int32_t n,
                                                          int shift, int dbits,
                                                          const int32_t *hist_scan,
                                                          uint32_t *keys_out, int32_t *vals_out) {
    __shared__ int wcount[kWaves][kRadixBins];
    __shared__ int gbase[kRadixBins];
    const int bins = 1 << dbits;
    const uint32_t mask = uint32_t(bins) - 1u;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    for (int d = threadIdx.x; d < bins; d += kBlock) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) wcount[w][d] = 0;
        gbase[d] = hist_scan[int64_t(d) * gridDim.x + blockIdx.x];
    }
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
        const uint32_t digit = (key[k] >> shift) & mask;
        uint64_t same = __ballot(valid);
#pragma unroll
        for (int b = 0; b < kRadixBits; ++b) {
            if (b < dbits) {   // uniform over the workgroup
                const bool bit = (digit >> b) & 1u;
                const uint64_t ones = __ballot(bit);
                same &= bit ? ones : ~ones;
            }
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
    for (int d = threadIdx.x; d < bins; d += kBlock) {
        int run = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const int c = wcount[w][d];
            wcount[w][d] = run;
            run += c;
        }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = base + int64_t(k) * kWaveSize + lane;
        if (i < n) {
            const uint32_t digit = (key[k] >> shift) & mask;
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

// Counters shared by the whole grid (counts, maxima) are reduced in the
// workgroup first and updated by one atomic per workgroup, and the kernels
// that update them run a capped grid over their elements: atomics on one
// address are performed one after another, so one per wave (what the
// compiler makes of per-thread updates) would cost tens of microseconds.
constexpr int kReduceBlocks = 256;

// Workgroup sum (MAX: maximum) of one value per thread; every thread of the
// workgroup calls it, the result is valid in thread 0. s_red holds kWaves
// words and is not reused by another call before a barrier.
template <bool MAX>
__device__ __forceinline__ int32_t block_reduce(int32_t v, int32_t *s_red) {
#pragma unroll
    for (int o = kWaveSize / 2; o > 0; o >>= 1) {
        const int32_t u = __shfl_xor(v, o, kWaveSize);
        v = MAX ? max(v, u) : v + u;
    }
    if ((threadIdx.x & (kWaveSize - 1)) == 0) s_red[threadIdx.x / kWaveSize] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 1; w < kWaves; ++w) v = MAX ? max(v, s_red[w]) : v + s_red[w];
    }
    return v;
}

// Non-empty cells and the largest interval into stats[0..1], the kept
// count (cell_start[n_cells]) into stats[10]; clears two per-cell arrays
// (the combo walk's counters) on the way.
__global__ __launch_bounds__(kBlock) void k_cell_stats(const int32_t *cell_start, int32_t n_cells,
                                                       int32_t *stats /* nonempty, max */,
                                                       int32_t *clear_a, int32_t *clear_b) {
    __shared__ int32_t s_n[kWaves], s_m[kWaves];
    if (blockIdx.x == 0 && threadIdx.x == 0) stats[10] = cell_start[n_cells];
    int32_t nonempty = 0, most = 0;
    for (int32_t c = blockIdx.x * kBlock + threadIdx.x; c < n_cells; c += gridDim.x * kBlock) {
        clear_a[c] = 0;
        clear_b[c] = 0;
        const int32_t cnt = cell_start[c + 1] - cell_start[c];
        nonempty += cnt > 0 ? 1 : 0;
        most = max(most, cnt);
    }
    nonempty = block_reduce<false>(nonempty, s_n);
    most = block_reduce<true>(most, s_m);
    if (threadIdx.x == 0) {
        if (nonempty > 0) atomicAdd(&stats[0], nonempty);
        if (most > 0) atomicMax(&stats[1], most);
    }
}


// ---------------------------------------------------------------- work partition
//
// Combos, items and cell classes as described in internal.h. Every kernel
// below is a plain per-element pass; ordering comes from scans and the
// stable radix sort only, so the partition is deterministic.

__global__ __launch_bounds__(kBlock) void k_fill(int32_t *p, int64_t n, int32_t v) {
    const int64_t i = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (i < n) p[i] = v;
}

struct ComboArgs {
    const int32_t *cell_of_point;
    int32_t N, D, H, W;
    int32_t allow_clean;        // 0 when rows do not fit the packed row range
    int32_t *combo_cell;        // [N*D*W]: cell of a clean combo, -1 none kept, -2 not clean
    int32_t *combo_range;       // [N*D*W]: h_lo | h_hi << 16
    int32_t *cell_generic;      // [n_cells]: 1 if a combo that is not clean touches the cell
    int32_t *cell_ncombo;       // [n_cells]: row segments of column-served combos in the cell
    int32_t planes;             // segments a combo may have and stay column-served
    int32_t *seg_cell;          // [planes][N*D*W]: cell of segment s of the combo, or -1
    int32_t *seg_range;         // [planes][N*D*W]: its rows h_lo | h_hi << 16
    int32_t *max_seg;           // most segments of a column-served combo
    int32_t *served_pts;        // kept points of column-served combos
    int32_t *class_counters;    // [2]: k_cell_class's counters, cleared here for it
};

// One thread per combo walks its H rows and splits the kept ones into
// segments: maximal runs of consecutive kept rows in one cell. A combo with
// at most `planes` segments is served by the column items, one segment per
// pass (a level camera gives every combo one segment: a clean combo);
// otherwise its cells are generic. The rows are loaded kWalkRows at a time
// before they are walked (rows past H read row H - 1 and count as dropped),
// so one round trip serves kWalkRows rows.
constexpr int kWalkRows = 16;

__device__ __forceinline__ void walk_rows(const ComboArgs &a, int64_t base, int32_t h0,
                                          int32_t (&cc)[kWalkRows]) {
#pragma unroll
    for (int u = 0; u < kWalkRows; ++u)
        cc[u] = a.cell_of_point[base + int64_t(min(h0 + u, a.H - 1)) * a.W];
}

__device__ __forceinline__ void combo_walk_one(const ComboArgs &a, int32_t X, int64_t n_combo,
                                               int32_t &max_seg, int32_t &served_pts) {
    const int32_t w = X % a.W, nd = X / a.W;
    const int64_t base = int64_t(nd) * a.H * a.W + w;
    int32_t cell[kMaxSeg], lo[kMaxSeg], hi[kMaxSeg];
    int32_t n_seg = 0, cur = -1, first = -1, last = -1, kept = 0;
    for (int32_t h0 = 0; h0 < a.H; h0 += kWalkRows) {
        int32_t cc[kWalkRows];
        walk_rows(a, base, h0, cc);
#pragma unroll
        for (int u = 0; u < kWalkRows; ++u) {
            const int32_t h = h0 + u;
            const int32_t c = h < a.H ? cc[u] : -1;
            if (c < 0) {
                cur = -1;
            } else {
                ++kept;
                if (first < 0) first = h;
                last = h;
                if (c != cur) {
                    if (n_seg < a.planes) {
                        cell[n_seg] = c;
                        lo[n_seg] = h;
                    }
                    ++n_seg;
                    cur = c;
                }
                if (n_seg <= a.planes) hi[n_seg - 1] = h + 1;
            }
        }
    }
    for (int s = 0; s < a.planes; ++s) a.seg_cell[int64_t(s) * n_combo + X] = -1;
    if (n_seg == 0) {
        a.combo_cell[X] = -1;
        a.combo_range[X] = 0;
        return;
    }
    if (a.allow_clean && n_seg <= a.planes) {
        for (int s = 0; s < n_seg; ++s) {
            a.seg_cell[int64_t(s) * n_combo + X] = cell[s];
            a.seg_range[int64_t(s) * n_combo + X] = lo[s] | (hi[s] << 16);
            atomicAdd(&a.cell_ncombo[cell[s]], 1);
        }
        max_seg = max(max_seg, n_seg);
        served_pts += kept;
        a.combo_cell[X] = n_seg == 1 ? cell[0] : -2;
        a.combo_range[X] = n_seg == 1 ? (lo[0] | (hi[0] << 16)) : 0;
    } else {
        a.combo_cell[X] = -2;
        a.combo_range[X] = 0;
        for (int32_t h0 = first; h0 <= last; h0 += kWalkRows) {
            int32_t cc[kWalkRows];
            walk_rows(a, base, h0, cc);
#pragma unroll
            for (int u = 0; u < kWalkRows; ++u)
                if (h0 + u <= last && cc[u] >= 0) atomicOr(&a.cell_generic[cc[u]], 1);
        }
    }
}

__global__ __launch_bounds__(kBlock) void k_combo_walk(ComboArgs a) {
    __shared__ int32_t s_m[kWaves], s_p[kWaves];
    if (blockIdx.x == 0 && threadIdx.x < 2) a.class_counters[threadIdx.x] = 0;
    const int64_t n_combo = int64_t(a.N) * a.D * a.W;
    int32_t max_seg = 0, served_pts = 0;
    for (int64_t x = int64_t(blockIdx.x) * kBlock + threadIdx.x; x < n_combo;
         x += int64_t(gridDim.x) * kBlock)
        combo_walk_one(a, int32_t(x), n_combo, max_seg, served_pts);
    max_seg = block_reduce<true>(max_seg, s_m);
    served_pts = block_reduce<false>(served_pts, s_p);
    if (threadIdx.x == 0) {
        if (max_seg > 0) atomicMax(a.max_seg, max_seg);
        if (served_pts > 0) atomicAdd(a.served_pts, served_pts);
    }
}

// Per cell: generic flag, empty flag (both arrays n_cells + 1 long, the
// last entry 0); counters[0] += column-served cells, counters[1] += heavy
// generic cells.
__global__ __launch_bounds__(kBlock) void k_cell_class(ComboArgs a, const int32_t *cell_start,
                                                       int32_t n_cells, int32_t *generic_flag,
                                                       int32_t *empty_flag, int32_t *counters) {
    __shared__ int32_t s_s[kWaves], s_h[kWaves];
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        generic_flag[n_cells] = 0;   // the flags are scanned over n_cells + 1 entries
        empty_flag[n_cells] = 0;
    }
    int32_t n_served = 0, n_heavy = 0;
    for (int32_t c = blockIdx.x * kBlock + threadIdx.x; c < n_cells; c += gridDim.x * kBlock) {
        const int32_t cnt = cell_start[c + 1] - cell_start[c];
        const bool served = cnt > 0 && a.cell_generic[c] == 0;
        generic_flag[c] = (cnt > 0 && !served) ? 1 : 0;
        empty_flag[c] = cnt == 0 ? 1 : 0;
        n_served += served ? 1 : 0;
        n_heavy += (cnt > kGenHeavy && !served) ? 1 : 0;
    }
    n_served = block_reduce<false>(n_served, s_s);
    n_heavy = block_reduce<false>(n_heavy, s_h);
    if (threadIdx.x == 0) {
        if (n_served > 0) atomicAdd(&counters[0], n_served);
        if (n_heavy > 0) atomicAdd(&counters[1], n_heavy);
    }
}

// Column table entries, one plane per segment index, and a flag on each
// segment of a cell fed by several segments (one more entry, 0, ends the
// flags).
__global__ __launch_bounds__(kBlock) void k_combo_table(ComboArgs a, int2 *table, int32_t *multi_flag) {
    const int64_t t = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    const int64_t n = int64_t(a.planes) * a.N * a.D * a.W;
    if (t == 0) multi_flag[n] = 0;   // scanned over n + 1 entries
    if (t >= n) return;
    const int32_t c = a.seg_cell[t];
    int2 e = make_int2(-1, 0);
    bool multi = false;
    if (c >= 0 && a.cell_generic[c] == 0) {
        multi = a.cell_ncombo[c] > 1;
        e = make_int2(c, a.seg_range[t] | int32_t(multi ? kComboMulti : 0u));
    }
    table[t] = e;
    multi_flag[t] = multi ? 1 : 0;
}

// Every entry of the column table empty ({-1, 0}): planes that the final
// partition does not use hold no stale entries.
__global__ __launch_bounds__(kBlock) void k_clear_table(int2 *table, int64_t n) {
    const int64_t t = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (t < n) table[t] = make_int2(-1, 0);
}

// Planes in use: one past the highest plane of the column table that holds
// an entry.
__global__ __launch_bounds__(kBlock) void k_planes_used(const int2 *table, int64_t n,
                                                        int32_t n_combo, int32_t *planes) {
    __shared__ int32_t s_m[kWaves];
    int32_t most = 0;
    for (int64_t t = int64_t(blockIdx.x) * kBlock + threadIdx.x; t < n; t += int64_t(gridDim.x) * kBlock)
        if (table[t].x >= 0) most = max(most, int32_t(t / n_combo) + 1);
    most = block_reduce<true>(most, s_m);
    if (threadIdx.x == 0 && most > 0) atomicMax(planes, most);
}

// Clean combos by pixel column: entry (n, w, d) = {cell, rows} of combo
// (n, d, w) when it is clean and its backward block holds no combo that is
// not clean, else {-1, 0} (such blocks are left to the per-row kernel).
__global__ __launch_bounds__(kBlock) void k_combo_cols(const int32_t *combo_cell,
                                                       const int32_t *combo_range,
                                                       const int32_t *mixed, int32_t n_combo,
                                                       int32_t W, int32_t D, int32_t blocks_w,
                                                       int2 *cols) {
    const int32_t x = blockIdx.x * kBlock + threadIdx.x;
    if (x >= n_combo) return;
    const int32_t w = x % W, nd = x / W, d = nd % D, n = nd / D;
    const int32_t c = combo_cell[x];
    const bool clean = c >= 0 && mixed[n * blocks_w + w / kBwdBlockCols] == 0;
    cols[(int64_t(n) * W + w) * D + d] = clean ? make_int2(c, combo_range[x]) : make_int2(-1, 0);
}

// Backward blocks (kBwdBlockCols pixel columns of one camera) that hold a
// combo that is not clean: flagged 1 (every writer stores the same value).
// One workgroup per backward block (camera n, kBwdBlockCols pixel columns):
// flags[block] = 1 when one of its combos is not clean, and *count adds the
// flagged blocks.
__global__ __launch_bounds__(kBlock) void k_bwd_blocks(const int32_t *combo_cell, int32_t W,
                                                       int32_t D, int32_t blocks_w, int32_t *flags,
                                                       int32_t *count) {
    __shared__ int32_t s_m[kWaves];
    const int32_t n = blockIdx.x / blocks_w, w0 = (blockIdx.x % blocks_w) * kBwdBlockCols;
    int32_t mixed = 0;
    for (int32_t i = threadIdx.x; i < D * kBwdBlockCols; i += kBlock) {
        const int32_t d = i / kBwdBlockCols, w = w0 + i % kBwdBlockCols;
        if (w < W && combo_cell[(int64_t(n) * D + d) * W + w] == -2) mixed = 1;
    }
    mixed = block_reduce<true>(mixed, s_m);
    if (threadIdx.x == 0) {
        flags[blockIdx.x] = mixed;
        if (mixed) atomicAdd(count, 1);
    }
}

// Not enough empty rows to hold the partial sums: cells fed by several
// combos become generic.
__global__ __launch_bounds__(kBlock) void k_demote_multi(ComboArgs a, int32_t n_cells) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c < 2) a.class_counters[c] = 0;
    if (c < n_cells && a.cell_generic[c] == 0 && a.cell_ncombo[c] > 1) a.cell_generic[c] = 1;
}

__global__ __launch_bounds__(kBlock) void k_empty_list(const int32_t *empty_pos, int32_t n_cells,
                                                       int32_t *empty_cells) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c < n_cells && empty_pos[c + 1] != empty_pos[c]) empty_cells[empty_pos[c]] = c;
}

// Segments of multi-segment cells as (cell, segment) pairs in segment order.
__global__ __launch_bounds__(kBlock) void k_multi_compact(const int32_t *seg_cell,
                                                          const int32_t *multi_pos, int32_t n_seg,
                                                          uint32_t *key, int32_t *val) {
    const int32_t X = blockIdx.x * kBlock + threadIdx.x;
    if (X >= n_seg || multi_pos[X + 1] == multi_pos[X]) return;
    key[multi_pos[X]] = uint32_t(seg_cell[X]);
    val[multi_pos[X]] = X;
}

// After the stable sort by cell, position i is the partial-sum slot of combo
// val[i]: a cell's slots are contiguous and in combo order. Slot i is kept in
// the BEV row of empty cell i (the output has a row for every cell, and the
// rows of empty cells are free until they are zeroed), so the table entry of
// the combo names that row; cell heads are flagged.
__global__ __launch_bounds__(kBlock) void k_multi_slots(const uint32_t *key, const int32_t *val,
                                                        int32_t n, const int32_t *empty_cells,
                                                        int2 *table, int32_t *head_flag) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i == 0) head_flag[n] = 0;   // scanned over n + 1 entries
    if (i >= n) return;
    table[val[i]].x = empty_cells[i];
    head_flag[i] = (i == 0 || key[i] != key[i - 1]) ? 1 : 0;
}

__global__ __launch_bounds__(kBlock) void k_multi_cells(const uint32_t *key, const int32_t *head_scan,
                                                        int32_t n, int32_t *multi_begin,
                                                        int32_t *multi_cell) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i > n) return;
    if (i == n) {
        multi_begin[head_scan[n]] = n;
        return;
    }
    if (head_scan[i + 1] != head_scan[i]) {
        multi_begin[head_scan[i]] = i;
        multi_cell[head_scan[i]] = int32_t(key[i]);
    }
}

// The borrowed rows of the first kCombineInline slots of each multi-combo
// cell, next to each other, so that the combine kernel finds them with one
// access; -1 past the cell's last slot. One thread per entry.
__global__ __launch_bounds__(kBlock) void k_multi_rows(const int32_t *multi_begin, int32_t n_multi,
                                                       const int32_t *empty_cells,
                                                       int32_t *multi_rows) {
    const int64_t x = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (x >= int64_t(n_multi) * kCombineInline) return;
    const int32_t k = int32_t(x / kCombineInline), u = int32_t(x % kCombineInline);
    const int32_t s = multi_begin[k] + u;
    multi_rows[x] = s < multi_begin[k + 1] ? empty_cells[s] : -1;
}

// Generic cells keyed for a descending sort by point count.
__global__ __launch_bounds__(kBlock) void k_compact_generic(const int32_t *cell_start, int32_t n_cells,
                                                            const int32_t *generic_pos,
                                                            int32_t max_per_cell, uint32_t *gen_key,
                                                            int32_t *gen_cell) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c >= n_cells || generic_pos[c + 1] == generic_pos[c]) return;
    gen_key[generic_pos[c]] = uint32_t(max_per_cell - (cell_start[c + 1] - cell_start[c]));
    gen_cell[generic_pos[c]] = c;
}

// 1 where a kept point of a generic cell starts a run: its previous depth
// bin (same pixel) is not a point of the same cell (one more entry, 0, ends
// the flags).
__global__ __launch_bounds__(kBlock) void k_run_flags(const int32_t *sorted_point, int32_t n_kept,
                                                      const int32_t *cell_of_point,
                                                      const int32_t *generic_pos, int32_t HW,
                                                      FastDiv div_hw, FastDiv div_d, int32_t D,
                                                      int32_t *flag) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i == 0) flag[n_kept] = 0;   // scanned over n_kept + 1 entries
    if (i >= n_kept) return;
    const int32_t p = sorted_point[i];
    const int32_t c = cell_of_point[p];
    const bool generic = generic_pos[c + 1] != generic_pos[c];
    const uint32_t q = fdiv(uint32_t(p), div_hw);
    const int32_t d = int32_t(q) - int32_t(fdiv(q, div_d)) * D;
    flag[i] = (generic && (d == 0 || cell_of_point[p - HW] != c)) ? 1 : 0;
}

// Runs per listed generic cell (one more entry, 0, for the scan), and each
// cell's list position.
__global__ __launch_bounds__(kBlock) void k_generic_counts(const int32_t *gen_cell, int32_t n_gen,
                                                           const int32_t *cell_start,
                                                           const int32_t *run_scan,
                                                           int32_t *runs_of, int32_t *pos_of_cell) {
    const int32_t k = blockIdx.x * kBlock + threadIdx.x;
    if (k == 0) runs_of[n_gen] = 0;   // scanned over n_gen + 1 entries
    if (k >= n_gen) return;
    const int32_t c = gen_cell[k];
    runs_of[k] = run_scan[cell_start[c + 1]] - run_scan[cell_start[c]];
    pos_of_cell[c] = k;
}

__global__ __launch_bounds__(kBlock) void k_generic_hdr(const int32_t *gen_cell, int32_t n_gen,
                                                        const int32_t *cell_start,
                                                        const int32_t *run_begin, int4 *hdr) {
    const int32_t k = blockIdx.x * kBlock + threadIdx.x;
    if (k >= n_gen) return;
    const int32_t c = gen_cell[k];
    hdr[k] = make_int4(c, run_begin[k], run_begin[k + 1] - run_begin[k],
                       cell_start[c + 1] - cell_start[c]);
}

// One thread per run start: the run's record, at its place in list order.
__global__ __launch_bounds__(kBlock) void k_generic_runs(const int32_t *sorted_point, int32_t n_kept,
                                                         const int32_t *cell_of_point,
                                                         const int32_t *cell_start,
                                                         const int32_t *run_scan,
                                                         const int32_t *pos_of_cell,
                                                         const int32_t *run_begin, int32_t HW,
                                                         int32_t D, FastDiv div_hw, FastDiv div_d,
                                                         int4 *runs) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n_kept || run_scan[i + 1] == run_scan[i]) return;
    const int32_t p = sorted_point[i];
    const int32_t c = cell_of_point[p];
    const uint32_t q = fdiv(uint32_t(p), div_hw);           // n * D + d
    const int32_t n = int32_t(fdiv(q, div_d));
    const int32_t d = int32_t(q) - n * D;
    const int32_t pixel = n * HW + (p - int32_t(q) * HW);
    int32_t len = 1;
    while (d + len < D && cell_of_point[p + len * HW] == c) ++len;
    const int32_t r = run_begin[pos_of_cell[c]] + (run_scan[i] - run_scan[cell_start[c]]);
    runs[r] = make_int4(p, pixel, len, 0);
}

int blocks_for(int64_t n) { return int((n + kBlock - 1) / kBlock); }
// Grid of a kernel that reduces into shared counters (at least one workgroup).
int reduce_blocks(int64_t n) { return std::max(1, std::min(blocks_for(n), kReduceBlocks)); }

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

// One device allocation carved into the plan build's temporaries: each
// piece is rounded to 256 bytes, and the total is reserved from upper bounds
// that the geometry fixes, so a build makes one allocation for them instead
// of one per array (each hipMalloc and hipFree costs about 10 us of host
// time).
struct Arena {
    char *base = nullptr;
    size_t cap = 0, used = 0;
    static size_t piece(size_t bytes) { return ((bytes ? bytes : 1) + 255) & ~size_t(255); }
    template <typename T>
    int take(T **p, size_t count, const char *what) {
        const size_t b = piece(count * sizeof(T));
        if (used + b > cap) {
            *p = nullptr;
            return bevpool_fail(BEVPOOL_ERR_HIP, "plan temporaries: %s does not fit the reserved %zu bytes",
                                what, cap);
        }
        *p = reinterpret_cast<T *>(base + used);
        used += b;
        return BEVPOOL_OK;
    }
};

// Chunk sums a multi-block scan of n elements needs.
int64_t scan_sums_needed(int64_t n) { return (n + kScanChunk - 1) / kScanChunk; }

// Exclusive scan of data[0..n) in place; *total receives the sum. sums:
// scratch of scan_sums_needed(n) ints (unused for a single chunk).
void device_scan(int32_t *data, int64_t n, int32_t *total, int32_t *sums, hipStream_t stream) {
    const int64_t nb = scan_sums_needed(n);
    if (nb <= kScanOneBlockChunks) {   // one launch: the workgroup walks the chunks
        hipLaunchKernelGGL(k_scan, dim3(1), dim3(kScanBlock), 0, stream, data, n, total);
        return;
    }
    hipLaunchKernelGGL(k_scan_sums, dim3(uint32_t(nb)), dim3(kScanBlock), 0, stream, data, n, sums);
    hipLaunchKernelGGL(k_scan, dim3(1), dim3(kScanBlock), 0, stream, sums, nb, total);
    hipLaunchKernelGGL(k_scan_apply, dim3(uint32_t(nb)), dim3(kScanBlock), 0, stream, data, n, sums);
}

}  // namespace
}  // namespace bevpool

using namespace bevpool;

int bevpool_build_plan(const double *intrinsics, const double *extrinsics,
                       const int32_t *host_cells, const bevpool_geometry &g, int32_t nz,
                       hipStream_t stream, bevpool_plan_s *plan) {
    const int64_t np64 = int64_t(g.n_cams) * g.n_depth * g.feat_h * g.feat_w;
    const int32_t np = int32_t(np64);
    const int32_t n_cells = g.nx * g.ny * nz;
    const int32_t N = g.n_cams, D = g.n_depth, H = g.feat_h, W = g.feat_w;
    const int32_t HW = H * W;
    const int64_t n_combo = int64_t(N) * D * W;
    // column-table planes: segment indices a combo may use (a segment has a
    // row of its own, so never more than H)
    const int32_t planes = H < kMaxSeg ? H : kMaxSeg;
    const int64_t n_seg = int64_t(planes) * n_combo;   // table entries reserved
    int64_t n_seg_act = n_seg;                          // entries of the planes in use
    plan->n_points = np64;
    plan->n_cells = n_cells;
    plan->nz = nz;

    int rc;
    if ((rc = dev_alloc(&plan->cell_of_point, size_t(np), "cell_of_point"))) return rc;
    if ((rc = dev_alloc(&plan->sorted_point, size_t(np), "sorted_point"))) return rc;
    if ((rc = dev_alloc(&plan->cell_start, size_t(n_cells) + 1, "cell_start"))) return rc;
    if ((rc = dev_alloc(&plan->column_table, size_t(n_seg), "column_table"))) return rc;

    // temporaries, carved from one arena that is freed on every exit path below
    const int64_t sort_cap = np64 > n_cells ? np64 : int64_t(n_cells);
    const int sort_tiles_cap = int((sort_cap + kSortTile - 1) / kSortTile);
    Arena arena;
    double *d_calib = nullptr;
    uint32_t *keys_a = nullptr, *keys_b = nullptr;
    int32_t *vals_a = nullptr, *vals_b = nullptr, *hist = nullptr, *small = nullptr;
    int32_t *scan_sums = nullptr;
    int32_t *flag_a = nullptr, *flag_b = nullptr;
    int32_t *combo_cell = nullptr, *combo_range = nullptr, *combo_flag = nullptr;
    int32_t *cell_generic = nullptr, *cell_ncombo = nullptr, *head_scan = nullptr;
    int32_t *run_scan = nullptr, *run_begin = nullptr, *pos_of_cell = nullptr;
    auto cleanup = [&]() { (void)hipFree(arena.base); };

    // Stable LSD radix sort of n (key, value) pairs on the keys' low `bits`
    // bits (radix_passes passes of radix_digit_bits bits), ping-ponging
    // between keys / kalt and vals / valt; keys and vals are left pointing at
    // the buffers that hold the result (vals ends in valt after an odd number
    // of passes).
    auto radix_sort = [&](uint32_t *&keys, uint32_t *kalt, int32_t *&vals, int32_t *valt, int32_t n,
                          int bits) -> int {
        if (n <= 0) return BEVPOOL_OK;
        const int tiles = int((int64_t(n) + kSortTile - 1) / kSortTile);
        const int passes = radix_passes(bits), dbits = radix_digit_bits(bits);
        uint32_t *kin = keys, *kout = kalt;
        int32_t *vin = vals, *vout = valt;
        for (int pass = 0; pass < passes; ++pass) {
            const int shift = dbits * pass;
            hipLaunchKernelGGL(k_radix_hist, dim3(tiles), dim3(kBlock), 0, stream, kin, n, shift,
                               dbits, hist);
            device_scan(hist, int64_t(tiles) << dbits, small + 3, scan_sums, stream);
            hipLaunchKernelGGL(k_radix_scatter, dim3(tiles), dim3(kBlock), 0, stream, kin, vin, n,
                               shift, dbits, hist, kout, vout);
            BEVPOOL_HIP(hipGetLastError());
            std::swap(kin, kout);
            std::swap(vin, vout);
        }
        keys = kin;
        vals = vin;
        return BEVPOOL_OK;
    };
    auto bits_for = [](int64_t max_key) {
        int b = 1;
        while ((int64_t(1) << b) <= max_key) ++b;
        return b;
    };
    auto fill = [&](int32_t *p, int64_t n, int32_t v) {
        if (n > 0) hipLaunchKernelGGL(k_fill, dim3(blocks_for(n)), dim3(kBlock), 0, stream, p, n, v);
    };
    auto to_host = [&](int32_t *dst, const int32_t *src) -> int {
        BEVPOOL_HIP(hipMemcpyAsync(dst, src, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
        return BEVPOOL_OK;
    };

    auto run = [&]() -> int {
        int rc2;
        {
            // upper bounds of every temporary taken below: the partial slots
            // (n_part) are at most the combos, the kept points at most the
            // points, the generic cells at most the cells
            const size_t i4 = sizeof(int32_t);
            const size_t sort_b = Arena::piece(size_t(sort_cap) * i4);
            const size_t cells1_b = Arena::piece((size_t(n_cells) + 1) * i4);
            const size_t combo1_b = Arena::piece((size_t(n_seg) + 1) * i4);
            arena.cap = Arena::piece(size_t(g.n_cams) * 16 * sizeof(double)) + 4 * sort_b +
                        Arena::piece(size_t(sort_tiles_cap) * kRadixBins * i4) + Arena::piece(16 * i4) +
                        Arena::piece(size_t(scan_sums_needed(sort_cap + 1)) * i4) +
                        5 * cells1_b +                 // flag_a, flag_b, cell_generic, cell_ncombo, run_begin
                        Arena::piece(size_t(n_cells) * i4) +          // pos_of_cell
                        2 * combo1_b +                 // combo_flag, head_scan
                        Arena::piece(size_t(n_combo) * i4) +          // combo_range
                        2 * Arena::piece(size_t(n_seg) * i4) +        // seg_cell, seg_range
                        Arena::piece((size_t(np) + 1) * i4);          // run_scan
            if ((rc2 = dev_alloc(&arena.base, arena.cap, "plan temporaries"))) return rc2;
        }
        const bool cal_in_args = g.n_cams <= kArgCams;
        if (!host_cells && !cal_in_args &&
            (rc2 = arena.take(&d_calib, size_t(g.n_cams) * 16, "calibration")))
            return rc2;
        if ((rc2 = arena.take(&keys_a, size_t(sort_cap), "sort keys"))) return rc2;
        if ((rc2 = arena.take(&keys_b, size_t(sort_cap), "sort keys"))) return rc2;
        if ((rc2 = arena.take(&vals_a, size_t(sort_cap), "sort values"))) return rc2;
        if ((rc2 = arena.take(&vals_b, size_t(sort_cap), "sort values"))) return rc2;
        if ((rc2 = arena.take(&hist, size_t(sort_tiles_cap) * kRadixBins, "radix histogram"))) return rc2;
        // [0..1] cell stats, [3] scan totals, [4..5] class counters, [6] most
        // segments of a combo, [7] their kept points, [8] generic cells, [9]
        // empty cells, [10] kept points, [11] segments of multi-combo cells,
        // [12] backward blocks with a combo that is not clean
        if ((rc2 = arena.take(&small, 16, "plan counters"))) return rc2;
        // the longest scan is over sort_cap + 1 elements (radix histograms
        // are shorter)
        if ((rc2 = arena.take(&scan_sums, size_t(scan_sums_needed(sort_cap + 1)), "scan chunk sums")))
            return rc2;
        if ((rc2 = arena.take(&flag_a, size_t(n_cells) + 1, "flags"))) return rc2;
        if ((rc2 = arena.take(&flag_b, size_t(n_cells) + 1, "flags"))) return rc2;

        fill(small, 16, 0);
        // the sort's point ids start in the buffer from which its passes end
        // in sorted_point (vals_b for an odd number of passes)
        const bool odd_passes = radix_passes(bits_for(n_cells)) % 2 == 1;
        int32_t *ids0 = odd_passes ? vals_b : plan->sorted_point;
        int32_t *ids1 = odd_passes ? plan->sorted_point : vals_b;
        if (host_cells) {
            // a stored association: the cell map as exported, checked by the caller
            BEVPOOL_HIP(hipMemcpyAsync(plan->cell_of_point, host_cells, sizeof(int32_t) * size_t(np),
                                       hipMemcpyHostToDevice, stream));
            hipLaunchKernelGGL(k_keys_from_cells, dim3(blocks_for(np)), dim3(kBlock), 0, stream,
                               plan->cell_of_point, np, n_cells, keys_a, ids0);
        } else {
            ProjectArgs pa;
            if (cal_in_args) {
                // up to kArgCams cameras: no host-to-device copy
                pa.intr = pa.extr = nullptr;
                memcpy(pa.cal, intrinsics, sizeof(double) * 4 * g.n_cams);
                memcpy(pa.cal + 4 * g.n_cams, extrinsics, sizeof(double) * 12 * g.n_cams);
            } else {
                BEVPOOL_HIP(hipMemcpyAsync(d_calib, intrinsics, sizeof(double) * 4 * g.n_cams,
                                           hipMemcpyHostToDevice, stream));
                BEVPOOL_HIP(hipMemcpyAsync(d_calib + 4 * g.n_cams, extrinsics,
                                           sizeof(double) * 12 * g.n_cams, hipMemcpyHostToDevice,
                                           stream));
                pa.intr = d_calib;
                pa.extr = d_calib + 4 * g.n_cams;
            }

            // Sec. III-B, precomputation: cell of every point, then the points
            // sorted by (cell, id) and the interval table.
            pa.g = g;
            pa.div_w = make_fastdiv(uint32_t(W));
            pa.div_h = make_fastdiv(uint32_t(H));
            pa.div_d = make_fastdiv(uint32_t(D));
            pa.n_points = np;
            pa.n_cells = n_cells;
            pa.nz = nz;
            pa.cell_of_point = plan->cell_of_point;
            pa.keys = keys_a;
            pa.vals = ids0;
            hipLaunchKernelGGL(k_project, dim3(blocks_for(np)), dim3(kBlock), 0, stream, pa);
        }
        BEVPOOL_HIP(hipGetLastError());
        uint32_t *skeys = keys_a;
        int32_t *sids = ids0;
        if ((rc2 = radix_sort(skeys, keys_b, sids, ids1, np, bits_for(n_cells)))) return rc2;
        if (sids != plan->sorted_point)
            BEVPOOL_HIP(hipMemcpyAsync(plan->sorted_point, sids, sizeof(int32_t) * size_t(np),
                                       hipMemcpyDeviceToDevice, stream));
        hipLaunchKernelGGL(k_cell_start, dim3(blocks_for(int64_t(np) + 1)), dim3(kBlock), 0,
                           stream, skeys, np, n_cells, plan->cell_start);
        // per-cell counters of the combo walk, cleared by k_cell_stats
        if ((rc2 = arena.take(&cell_generic, size_t(n_cells), "cell classes"))) return rc2;
        if ((rc2 = arena.take(&cell_ncombo, size_t(n_cells), "cell combos"))) return rc2;
        hipLaunchKernelGGL(k_cell_stats, dim3(reduce_blocks(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, small, cell_generic, cell_ncombo);
        BEVPOOL_HIP(hipGetLastError());

        // combos, cell classes and the column table
        // the combo cells and rows stay with the plan (the backward pass
        // reads them)
        if ((rc2 = dev_alloc(&plan->combo_cells, size_t(n_combo), "combo cells"))) return rc2;
        combo_cell = plan->combo_cells;
        if ((rc2 = arena.take(&combo_range, size_t(n_combo), "combo ranges"))) return rc2;
        if ((rc2 = arena.take(&combo_flag, size_t(n_seg) + 1, "segment flags"))) return rc2;
        int32_t *seg_cell = nullptr, *seg_range = nullptr;
        if ((rc2 = arena.take(&seg_cell, size_t(n_seg), "segment cells"))) return rc2;
        if ((rc2 = arena.take(&seg_range, size_t(n_seg), "segment rows"))) return rc2;
        ComboArgs ca;
        ca.cell_of_point = plan->cell_of_point;
        ca.N = N;
        ca.D = D;
        ca.H = H;
        ca.W = W;
        ca.allow_clean = H < kMaxFeatH ? 1 : 0;
        ca.combo_cell = combo_cell;
        ca.combo_range = combo_range;
        ca.cell_generic = cell_generic;
        ca.cell_ncombo = cell_ncombo;
        ca.planes = planes;
        ca.seg_cell = seg_cell;
        ca.seg_range = seg_range;
        ca.max_seg = small + 6;
        ca.served_pts = small + 7;
        ca.class_counters = small + 4;
        // (k_combo_table writes every entry of every plane: no clearing first)
        hipLaunchKernelGGL(k_combo_walk, dim3(reduce_blocks(n_combo)), dim3(kBlock), 0, stream, ca);
        int32_t stats[4], counters[2], n_gen = 0, n_empty = 0, kept = 0, n_part = 0;
        // (the class counters small[4..5] are cleared by k_combo_walk or
        // k_demote_multi, which run before each classification)
        auto classify = [&]() -> int {
            hipLaunchKernelGGL(k_cell_class, dim3(reduce_blocks(n_cells)), dim3(kBlock), 0, stream, ca,
                               plan->cell_start, n_cells, flag_a, flag_b, small + 4);
            hipLaunchKernelGGL(k_combo_table, dim3(blocks_for(n_seg_act)), dim3(kBlock), 0, stream,
                               ca, plan->column_table, combo_flag);
            device_scan(flag_a, int64_t(n_cells) + 1, small + 8, scan_sums, stream);       // generic cells
            device_scan(flag_b, int64_t(n_cells) + 1, small + 9, scan_sums, stream);       // empty cells
            device_scan(combo_flag, n_seg_act + 1, small + 11, scan_sums, stream);  // segments of multi cells
            BEVPOOL_HIP(hipGetLastError());
            int32_t h[12];
            BEVPOOL_HIP(hipMemcpyAsync(h, small, sizeof(h), hipMemcpyDeviceToHost, stream));
            BEVPOOL_HIP(hipStreamSynchronize(stream));
            stats[0] = h[0];
            stats[1] = h[1];
            stats[2] = h[6];       // most segments of a column-served combo
            stats[3] = h[7];       // kept points of column-served combos
            counters[0] = h[4];
            counters[1] = h[5];
            n_gen = h[8];          // generic cells
            n_empty = h[9];        // empty cells
            kept = h[10];          // kept points (k_cell_stats)
            n_part = h[11];        // combos of multi-combo cells (partial slots)
            return BEVPOOL_OK;
        };
        if ((rc2 = classify())) return rc2;
        if (ca.planes > 1 && int64_t(stats[3]) * 2 < int64_t(kept)) {
            // segments serve under half of the kept points (a strongly tilted
            // rig): the extra passes would cost more than they save, so the
            // partition is rebuilt with whole combos only
            ca.planes = 1;
            n_seg_act = n_combo;
            hipLaunchKernelGGL(k_clear_table, dim3(blocks_for(n_seg)), dim3(kBlock), 0, stream,
                               plan->column_table, n_seg);
            fill(cell_generic, n_cells, 0);
            fill(cell_ncombo, n_cells, 0);
            fill(small + 6, 2, 0);
            hipLaunchKernelGGL(k_combo_walk, dim3(reduce_blocks(n_combo)), dim3(kBlock), 0, stream, ca);
            if ((rc2 = classify())) return rc2;
        }
        if (n_part > n_empty) {
            hipLaunchKernelGGL(k_demote_multi, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream, ca,
                               n_cells);
            if ((rc2 = classify())) return rc2;
        }
        plan->n_nonempty = stats[0];
        plan->max_per_cell = stats[1];
        plan->n_kept = kept;
        plan->n_column = counters[0];
        plan->n_generic_heavy = counters[1];
        plan->n_generic = n_gen;
        plan->n_empty = n_empty;
        plan->n_partials = n_part;
        // planes in use, from the final table (cells demoted to generic leave
        // their segments' planes empty)
        hipLaunchKernelGGL(k_planes_used, dim3(reduce_blocks(n_seg_act)), dim3(kBlock), 0, stream,
                           plan->column_table, n_seg_act, int32_t(n_combo), small + 2);

        // the backward blocks holding a combo that is not clean, and the clean
        // combos of the other blocks by pixel column
        const int32_t bwd_bw = (W + kBwdBlockCols - 1) / kBwdBlockCols;
        plan->n_bwd_blocks = N * bwd_bw;
        if ((rc2 = dev_alloc(&plan->bwd_mixed, size_t(plan->n_bwd_blocks), "backward blocks")))
            return rc2;
        hipLaunchKernelGGL(k_bwd_blocks, dim3(plan->n_bwd_blocks), dim3(kBlock), 0, stream,
                           combo_cell, W, D, bwd_bw, plan->bwd_mixed, small + 12);
        if ((rc2 = dev_alloc(&plan->combo_cols, size_t(n_combo), "combos by column"))) return rc2;
        hipLaunchKernelGGL(k_combo_cols, dim3(blocks_for(n_combo)), dim3(kBlock), 0, stream,
                           combo_cell, combo_range, plan->bwd_mixed, int32_t(n_combo), W, D, bwd_bw,
                           plan->combo_cols);
        BEVPOOL_HIP(hipGetLastError());

        // cells without points, ascending
        if ((rc2 = dev_alloc(&plan->empty_cells, size_t(n_empty), "empty_cells"))) return rc2;
        hipLaunchKernelGGL(k_empty_list, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream, flag_b,
                           n_cells, plan->empty_cells);

        // partial-sum slots of the multi-combo cells, kept in the first
        // n_part empty rows
        if ((rc2 = arena.take(&head_scan, size_t(n_part) + 1, "multi heads"))) return rc2;
        uint32_t *mkeys = keys_a;
        int32_t *mvals = vals_a;
        if (n_part > 0) {
            hipLaunchKernelGGL(k_multi_compact, dim3(blocks_for(n_seg_act)), dim3(kBlock), 0, stream,
                               seg_cell, combo_flag, int32_t(n_seg_act), keys_a, vals_a);
            if ((rc2 = radix_sort(mkeys, keys_b, mvals, vals_b, n_part, bits_for(n_cells)))) return rc2;
            hipLaunchKernelGGL(k_multi_slots, dim3(blocks_for(n_part)), dim3(kBlock), 0, stream,
                               mkeys, mvals, n_part, plan->empty_cells, plan->column_table,
                               head_scan);
            // the number of multi-combo cells lands in small[3]
            device_scan(head_scan, int64_t(n_part) + 1, small + 3, scan_sums, stream);
        } else {
            fill(head_scan, 1, 0);
        }
        BEVPOOL_HIP(hipGetLastError());
        // one read-back for the counts that size the remaining arrays
        int32_t h[16];
        BEVPOOL_HIP(hipMemcpyAsync(h, small, sizeof(h), hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        const int32_t n_multi = n_part > 0 ? h[3] : 0;
        plan->n_bwd_mixed = h[12];
        plan->n_multi = n_multi;
        plan->n_planes = h[2] > 0 ? h[2] : 1;
        if ((rc2 = dev_alloc(&plan->multi_begin, size_t(n_multi) + 1, "multi_begin"))) return rc2;
        if ((rc2 = dev_alloc(&plan->multi_cell, size_t(n_multi), "multi_cell"))) return rc2;
        if ((rc2 = dev_alloc(&plan->multi_rows, size_t(n_multi) * kCombineInline, "multi_rows")))
            return rc2;
        if ((rc2 = dev_alloc(&plan->generic_hdr, size_t(n_gen), "generic_hdr"))) return rc2;
        hipLaunchKernelGGL(k_multi_cells, dim3(blocks_for(int64_t(n_part) + 1)), dim3(kBlock), 0,
                           stream, mkeys, head_scan, n_part, plan->multi_begin, plan->multi_cell);
        if (n_multi > 0)
            hipLaunchKernelGGL(k_multi_rows, dim3(blocks_for(int64_t(n_multi) * kCombineInline)),
                               dim3(kBlock), 0, stream, plan->multi_begin, n_multi,
                               plan->empty_cells, plan->multi_rows);
        BEVPOOL_HIP(hipGetLastError());

        // generic cells by descending point count
        if (n_gen == 0) {
            // every cell with points is column-served (a level rig): no runs
            plan->n_runs = 0;
            if ((rc2 = dev_alloc(&plan->generic_runs, 0, "generic_runs"))) return rc2;
            BEVPOOL_HIP(hipGetLastError());
            BEVPOOL_HIP(hipStreamSynchronize(stream));
            return BEVPOOL_OK;
        }
        uint32_t *gen_key = keys_a;   // the sort buffers are free again after k_multi_cells
        int32_t *gen_cell = vals_a;
        hipLaunchKernelGGL(k_compact_generic, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, flag_a, plan->max_per_cell, gen_key, gen_cell);
        BEVPOOL_HIP(hipGetLastError());
        if ((rc2 = radix_sort(gen_key, keys_b, gen_cell, vals_b, n_gen, bits_for(plan->max_per_cell))))
            return rc2;

        // runs of the generic cells, in list order
        if ((rc2 = arena.take(&run_scan, size_t(kept) + 1, "run flags"))) return rc2;
        if ((rc2 = arena.take(&run_begin, size_t(n_gen) + 1, "run offsets"))) return rc2;
        if ((rc2 = arena.take(&pos_of_cell, size_t(n_cells), "cell positions"))) return rc2;
        const FastDiv div_hw = make_fastdiv(uint32_t(HW)), div_d = make_fastdiv(uint32_t(D));
        if (kept > 0)
            hipLaunchKernelGGL(k_run_flags, dim3(blocks_for(kept)), dim3(kBlock), 0, stream,
                               plan->sorted_point, kept, plan->cell_of_point, flag_a, HW, div_hw,
                               div_d, D, run_scan);
        device_scan(run_scan, int64_t(kept) + 1, small + 3, scan_sums, stream);
        if (n_gen > 0)
            hipLaunchKernelGGL(k_generic_counts, dim3(blocks_for(n_gen)), dim3(kBlock), 0, stream,
                               gen_cell, n_gen, plan->cell_start, run_scan, run_begin, pos_of_cell);
        device_scan(run_begin, int64_t(n_gen) + 1, small + 3, scan_sums, stream);
        if (n_gen > 0)
            hipLaunchKernelGGL(k_generic_hdr, dim3(blocks_for(n_gen)), dim3(kBlock), 0, stream,
                               gen_cell, n_gen, plan->cell_start, run_begin, plan->generic_hdr);
        BEVPOOL_HIP(hipGetLastError());
        int32_t n_runs;
        if ((rc2 = to_host(&n_runs, run_begin + n_gen))) return rc2;
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        plan->n_runs = n_runs;
        if ((rc2 = dev_alloc(&plan->generic_runs, size_t(n_runs), "generic_runs"))) return rc2;
        if (kept > 0)
            hipLaunchKernelGGL(k_generic_runs, dim3(blocks_for(kept)), dim3(kBlock), 0, stream,
                               plan->sorted_point, kept, plan->cell_of_point, plan->cell_start,
                               run_scan, pos_of_cell, run_begin, HW, D, div_hw, div_d,
                               plan->generic_runs);
        BEVPOOL_HIP(hipGetLastError());
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        return BEVPOOL_OK;
    };
    rc = run();
    if (rc != BEVPOOL_OK) (void)hipStreamSynchronize(stream);
    cleanup();
    return rc;
}

// ---------------------------------------------------------------- association without allocation
//
// bevpool_associate_noalloc: the association of the "Precomputation"
// paragraph (every point's cell, the points sorted by cell, the interval
// table) into caller buffers, for callers that cannot allocate. Its
// temporaries (the calibration, the radix sort's second key and value
// arrays, histograms, counters, scan sums) live in one file-scope device
// array of fixed size, which each device holds while the library is loaded.
// Host code never uses the array's name as an address: the device address
// comes from hipGetSymbolAddress, once per device, with that device current.
namespace bevpool {
namespace {

constexpr size_t scratch_piece(size_t b) { return (b + 255) & ~size_t(255); }
constexpr int64_t kAssocTiles = (kAssocMaxPoints + kSortTile - 1) / kSortTile;
constexpr int64_t kAssocSums = (kAssocTiles * kRadixBins + kScanChunk - 1) / kScanChunk;
constexpr size_t kOffCalib = 0;
constexpr size_t kOffKeysA = kOffCalib + scratch_piece(size_t(kAssocMaxCams) * 16 * sizeof(double));
constexpr size_t kOffKeysB = kOffKeysA + scratch_piece(size_t(kAssocMaxPoints) * 4);
constexpr size_t kOffValsB = kOffKeysB + scratch_piece(size_t(kAssocMaxPoints) * 4);
constexpr size_t kOffHist = kOffValsB + scratch_piece(size_t(kAssocMaxPoints) * 4);
constexpr size_t kOffSmall = kOffHist + scratch_piece(size_t(kAssocTiles) * kRadixBins * 4);
constexpr size_t kOffSums = kOffSmall + scratch_piece(16 * 4);
constexpr size_t kAssocScratchBytes = kOffSums + scratch_piece(size_t(kAssocSums) * 4);
static_assert(kAssocScratchBytes == kAssocScratchTotal, "scratch size stated in internal.h");

static __device__ __align__(256) char noalloc_scratch[kAssocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
char *g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch (looked up on first use).
int scratch_of_device(int dev, char **out) {
    if (dev < 0 || dev >= kMaxDevices)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "device %d is beyond the %d supported", dev,
                            kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        BEVPOOL_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch)));
        if (!p) return bevpool_fail(BEVPOOL_ERR_HIP, "no device address for the scratch array");
        g_scratch_ptr[dev] = static_cast<char *>(p);
    }
    *out = g_scratch_ptr[dev];
    return BEVPOOL_OK;
}

// The calibration travels in the kernel arguments, so the call reads the
// caller's host arrays before it returns and copies nothing from host memory.
struct CalibArgs {
    double v[kAssocMaxCams * 16];   // [N][4] intrinsics, then [N][12] extrinsics
    int32_t n;                      // values used
};
__global__ void k_store_calib(CalibArgs a, double *dst) {
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) dst[i] = a.v[i];
}

}  // namespace
}  // namespace bevpool

int bevpool_associate_into(const double *intrinsics, const double *extrinsics,
                           const bevpool_geometry &g, int32_t *cell_of_point,
                           int32_t *sorted_point, int32_t *cell_start, hipStream_t stream) {
    using namespace bevpool;
    const int64_t np64 = int64_t(g.n_cams) * g.n_depth * g.feat_h * g.feat_w;
    if (np64 > kAssocMaxPoints || g.n_cams > kAssocMaxCams)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG,
                            "%lld points on %d cameras exceed the no-allocation maximum of %lld points "
                            "on %d cameras", (long long)np64, g.n_cams, (long long)kAssocMaxPoints,
                            kAssocMaxCams);
    int dev = -1;
    BEVPOOL_HIP(hipGetDevice(&dev));
    char *base = nullptr;
    int rc = scratch_of_device(dev, &base);
    if (rc != BEVPOOL_OK) return rc;
    double *calib = reinterpret_cast<double *>(base + kOffCalib);
    uint32_t *keys_a = reinterpret_cast<uint32_t *>(base + kOffKeysA);
    uint32_t *keys_b = reinterpret_cast<uint32_t *>(base + kOffKeysB);
    int32_t *vals_b = reinterpret_cast<int32_t *>(base + kOffValsB);
    int32_t *hist = reinterpret_cast<int32_t *>(base + kOffHist);
    int32_t *small = reinterpret_cast<int32_t *>(base + kOffSmall);
    int32_t *sums = reinterpret_cast<int32_t *>(base + kOffSums);
    const int32_t np = int32_t(np64), n_cells = g.nx * g.ny;

    CalibArgs ca;
    ca.n = 16 * g.n_cams;
    for (int i = 0; i < 4 * g.n_cams; ++i) ca.v[i] = intrinsics[i];
    for (int i = 0; i < 12 * g.n_cams; ++i) ca.v[4 * g.n_cams + i] = extrinsics[i];
    hipLaunchKernelGGL(k_store_calib, dim3(1), dim3(kBlock), 0, stream, ca, calib);
    // counters start at zero on every call (the array keeps the last call's contents)
    hipLaunchKernelGGL(k_fill, dim3(1), dim3(kBlock), 0, stream, small, int64_t(16), 0);

    ProjectArgs pa;
    pa.intr = calib;
    pa.extr = calib + 4 * g.n_cams;
    pa.g = g;
    pa.div_w = make_fastdiv(uint32_t(g.feat_w));
    pa.div_h = make_fastdiv(uint32_t(g.feat_h));
    pa.div_d = make_fastdiv(uint32_t(g.n_depth));
    pa.n_points = np;
    pa.n_cells = n_cells;
    pa.nz = 1;
    // stable LSD radix sort of (cell, point id) on the cell's bits
    // (radix_passes passes); the ids start in the buffer from which the
    // passes end in sorted_point
    int bits = 1;
    while ((int64_t(1) << bits) <= int64_t(n_cells)) ++bits;
    const bool odd_passes = radix_passes(bits) % 2 == 1;
    pa.cell_of_point = cell_of_point;
    pa.keys = keys_a;
    pa.vals = odd_passes ? vals_b : sorted_point;
    hipLaunchKernelGGL(k_project, dim3(blocks_for(np)), dim3(kBlock), 0, stream, pa);
    BEVPOOL_HIP(hipGetLastError());

    const int tiles = int((int64_t(np) + kSortTile - 1) / kSortTile);
    uint32_t *kin = keys_a, *kout = keys_b;
    int32_t *vin = pa.vals, *vout = odd_passes ? sorted_point : vals_b;
    const int dbits = radix_digit_bits(bits);
    for (int shift = 0; shift < bits; shift += dbits) {
        hipLaunchKernelGGL(k_radix_hist, dim3(tiles), dim3(kBlock), 0, stream, kin, np, shift, dbits,
                           hist);
        device_scan(hist, int64_t(tiles) << dbits, small + 3, sums, stream);
        hipLaunchKernelGGL(k_radix_scatter, dim3(tiles), dim3(kBlock), 0, stream, kin, vin, np, shift,
                           dbits, hist, kout, vout);
        BEVPOOL_HIP(hipGetLastError());
        std::swap(kin, kout);
        std::swap(vin, vout);
    }
    if (vin != sorted_point)
        BEVPOOL_HIP(hipMemcpyAsync(sorted_point, vin, sizeof(int32_t) * size_t(np),
                                   hipMemcpyDeviceToDevice, stream));
    hipLaunchKernelGGL(k_cell_start, dim3(blocks_for(int64_t(np) + 1)), dim3(kBlock), 0, stream, kin,
                       np, n_cells, cell_start);
    BEVPOOL_HIP(hipGetLastError());
    return BEVPOOL_OK;
}
