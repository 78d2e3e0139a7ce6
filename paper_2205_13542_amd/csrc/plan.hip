// Plan building for BEV pooling: the camera-fixed point-to-cell association
// (BEVFusion, arXiv 2205.13542, Sec. III-B, "Precomputation" paragraph:
// compute each frustum point's 3-D coordinate and grid index once, sort the
// points by grid index and record their ranks).
//
// Kernels, in launch order:
//   k_project      one thread per point: camera ray -> ego frame -> cell id
//   k_radix_hist   } stable LSD radix sort of (cell, point id), 8-bit digits;
//   k_scan...      } input in id order, so ties stay in id order (scans:
//   k_radix_scatter} one workgroup for a short array, else chunk sums,
//                    their scan and per-chunk scans from the offsets)
//   k_cell_start   interval table from the sorted keys
//   k_cell_stats   non-empty cells and the largest interval
//   k_combo_walk ... k_generic_runs   work partition of the forward pass:
//                  clean combos, swept cells and the column table, empty
//                  cells, generic cells and their runs
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
constexpr int kScanChunk = kScanBlock * kScanItems;  // elements per workgroup of a multi-block scan
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

// Four single counts next to each other, so that one copy brings them to
// the host.
__global__ void k_gather4(int32_t *dst, const int32_t *a, const int32_t *b, const int32_t *c,
                          const int32_t *d) {
    dst[0] = *a;
    dst[1] = *b;
    dst[2] = *c;
    dst[3] = *d;
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
    int32_t sweep_ok;           // 0 when the camera width does not fit a sweep workgroup
    int32_t *combo_cell;        // [N*D*W]: cell of a clean combo, -1 none kept, -2 not clean
    int32_t *combo_range;       // [N*D*W]: h_lo | h_hi << 15
    int32_t *cell_generic;      // [n_cells]: 1 if a combo that is not clean touches the cell
    int32_t *cell_ncombo;       // [n_cells]: clean combos in the cell
    int32_t *cell_key_min;      // [n_cells]: smallest and largest n * D + d of its clean combos
    int32_t *cell_key_max;
    int32_t *cell_w_min;        // [n_cells]: first and last pixel column of its clean combos
    int32_t *cell_w_max;
};

// One thread per combo walks its H rows. A combo whose kept rows are
// consecutive and lie in one cell is clean; otherwise every cell it touches
// is generic.
__global__ __launch_bounds__(kBlock) void k_combo_walk(ComboArgs a) {
    const int64_t x = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    const int64_t n_combo = int64_t(a.N) * a.D * a.W;
    if (x >= n_combo) return;
    const int32_t X = int32_t(x);
    const int32_t w = X % a.W, nd = X / a.W;
    const int64_t base = int64_t(nd) * a.H * a.W + w;
    int32_t cell = -1, lo = 0, hi = 0, n_seg = 0, cur = -1, first = -1, last = -1;
    for (int32_t h = 0; h < a.H; ++h) {
        const int32_t c = a.cell_of_point[base + int64_t(h) * a.W];
        if (c < 0) {
            cur = -1;
            continue;
        }
        if (first < 0) first = h;
        last = h;
        if (c != cur) {
            if (n_seg == 0) {
                cell = c;
                lo = h;
            }
            ++n_seg;
            cur = c;
        }
        if (n_seg == 1) hi = h + 1;
    }
    if (n_seg == 0) {
        a.combo_cell[X] = -1;
        a.combo_range[X] = 0;
        return;
    }
    if (a.allow_clean && n_seg == 1) {
        a.combo_cell[X] = cell;
        a.combo_range[X] = lo | (hi << 15);
        const int32_t key = nd;   // n * D + d
        atomicAdd(&a.cell_ncombo[cell], 1);
        atomicMin(&a.cell_key_min[cell], key);
        atomicMax(&a.cell_key_max[cell], key);
        atomicMin(&a.cell_w_min[cell], w);
        atomicMax(&a.cell_w_max[cell], w);
    } else {
        a.combo_cell[X] = -2;
        a.combo_range[X] = 0;
        for (int32_t h = first; h <= last; ++h) {
            const int32_t c = a.cell_of_point[base + int64_t(h) * a.W];
            if (c >= 0) atomicOr(&a.cell_generic[c], 1);
        }
    }
}

// A cell with points is swept when no combo that is not clean touches it and
// its clean combos share one camera and depth bin and fill consecutive
// columns (the counts then match the column span).
__device__ __forceinline__ bool cell_swept(const ComboArgs &a, int32_t c) {
    return a.sweep_ok && a.cell_generic[c] == 0 && a.cell_ncombo[c] > 0 &&
           a.cell_key_min[c] == a.cell_key_max[c] &&
           a.cell_w_max[c] - a.cell_w_min[c] + 1 == a.cell_ncombo[c];
}

// Per cell: run-cell flag (a generic cell touched by a combo that is not
// clean: its points are gathered in runs), combo-cell flag (any other
// generic cell: all its points lie in clean combos, gathered combo by
// combo), empty flag; counters[0] += swept cells, counters[1] += heavy run
// cells, counters[2] += swept cells fed by several combos.
__global__ __launch_bounds__(kBlock) void k_cell_class(ComboArgs a, const int32_t *cell_start,
                                                       int32_t n_cells, int32_t *generic_flag,
                                                       int32_t *empty_flag, int32_t *combo_flag,
                                                       int32_t *counters) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c >= n_cells) return;
    const int32_t cnt = cell_start[c + 1] - cell_start[c];
    const bool swept = cnt > 0 && cell_swept(a, c);
    const bool by_combo = cnt > 0 && !swept && a.cell_generic[c] == 0;
    const bool by_run = cnt > 0 && !swept && !by_combo;
    generic_flag[c] = by_run ? 1 : 0;
    combo_flag[c] = by_combo ? 1 : 0;
    empty_flag[c] = cnt == 0 ? 1 : 0;
    if (swept) atomicAdd(&counters[0], 1);
    if (cnt > kGenHeavy && by_run) atomicAdd(&counters[1], 1);
    if (swept && a.cell_ncombo[c] > 1) atomicAdd(&counters[2], 1);
}

// The combos of combo cells, as (cell, combo) pairs in combo order: flag_x
// marks them, its scan places them.
__global__ __launch_bounds__(kBlock) void k_cc_flags(const int32_t *combo_cell, int64_t n_combo,
                                                     const int32_t *combo_flag, int32_t *flag_x) {
    const int64_t x = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (x > n_combo) return;
    const int32_t c = x < n_combo ? combo_cell[x] : -1;
    flag_x[x] = (c >= 0 && combo_flag[c + 1] != combo_flag[c]) ? 1 : 0;
}

__global__ __launch_bounds__(kBlock) void k_cc_compact(const int32_t *combo_cell, int64_t n_combo,
                                                       const int32_t *pos_x, uint32_t *key,
                                                       int32_t *val) {
    const int64_t x = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (x >= n_combo || pos_x[x + 1] == pos_x[x]) return;
    key[pos_x[x]] = uint32_t(combo_cell[x]);
    val[pos_x[x]] = int32_t(x);
}

// After the stable sort by cell: entry i is combo val[i] of cell key[i]; the
// combo list gets {combo, its rows h_lo | h_hi << 15} and each combo cell
// its header {cell, first entry, entries, points}. Combo cells are listed in
// cell order, which is the order of their first entries.
__global__ __launch_bounds__(kBlock) void k_cc_list(const uint32_t *key, const int32_t *val, int32_t n,
                                                    const int32_t *combo_range, const int32_t *combo_pos,
                                                    const int32_t *cell_start, int2 *list, int4 *hdr) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    list[i] = make_int2(val[i], combo_range[val[i]]);
    const uint32_t c = key[i];
    if (i == 0 || key[i - 1] != c) {
        int32_t e = i + 1;
        while (e < n && key[e] == c) ++e;
        hdr[combo_pos[c]] = make_int4(int32_t(c), i, e - i, cell_start[c + 1] - cell_start[c]);
    }
}

// Column-table entries: the combos of swept cells, with their row range and
// whether they are the first or last column of their cell. The table is
// kept as [N][W][D], so that the 16 depth bins that a sweep step reads at
// one column are adjacent.
__global__ __launch_bounds__(kBlock) void k_combo_table(ComboArgs a, int2 *table) {
    const int64_t t = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (t >= int64_t(a.N) * a.D * a.W) return;
    const int32_t w_ = int32_t(t % a.W), nd = int32_t(t / a.W);
    const int32_t n_ = nd / a.D, d_ = nd - n_ * a.D;
    const int64_t slot = (int64_t(n_) * a.W + w_) * a.D + d_;
    const int32_t c = a.combo_cell[t];
    int2 e = make_int2(-1, 0);
    if (c >= 0 && cell_swept(a, c)) {
        const int32_t w = int32_t(t % a.W);
        uint32_t y = uint32_t(a.combo_range[t]);
        if (w == a.cell_w_min[c]) y |= kColFirst;
        if (w == a.cell_w_max[c]) y |= kColLast;
        e = make_int2(c, int32_t(y));
    }
    table[slot] = e;
}

__global__ __launch_bounds__(kBlock) void k_empty_list(const int32_t *empty_pos, int32_t n_cells,
                                                       int32_t *empty_cells) {
    const int32_t c = blockIdx.x * kBlock + threadIdx.x;
    if (c < n_cells && empty_pos[c + 1] != empty_pos[c]) empty_cells[empty_pos[c]] = c;
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
// bin (same pixel) is not a point of the same cell.
__global__ __launch_bounds__(kBlock) void k_run_flags(const int32_t *sorted_point, int32_t n_kept,
                                                      const int32_t *cell_of_point,
                                                      const int32_t *generic_pos, int32_t HW,
                                                      FastDiv div_hw, FastDiv div_d, int32_t D,
                                                      int32_t *flag) {
    const int32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n_kept) return;
    const int32_t p = sorted_point[i];
    const int32_t c = cell_of_point[p];
    const bool generic = generic_pos[c + 1] != generic_pos[c];
    const uint32_t q = fdiv(uint32_t(p), div_hw);
    const int32_t d = int32_t(q) - int32_t(fdiv(q, div_d)) * D;
    flag[i] = (generic && (d == 0 || cell_of_point[p - HW] != c)) ? 1 : 0;
}

// Runs per listed generic cell, and each cell's list position.
__global__ __launch_bounds__(kBlock) void k_generic_counts(const int32_t *gen_cell, int32_t n_gen,
                                                           const int32_t *cell_start,
                                                           const int32_t *run_scan,
                                                           int32_t *runs_of, int32_t *pos_of_cell) {
    const int32_t k = blockIdx.x * kBlock + threadIdx.x;
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
    if (nb <= 1) {
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

// Rows of staged depth probabilities per pass of a sweep workgroup (a
// multiple of 4, one matrix-core step each), or 0 when a camera row of the
// given width does not fit the LDS buffer.
int bevpool_sweep_rows(int32_t W, int32_t H) {
    // the buffer holds kSweepDepths depth bins of r rows of W values, each
    // depth bin (r W) | 1 values long; 8 rows when a wave has at most 6
    // columns (the kernel's two instantiations: 6 columns and 2 steps of 4
    // rows, or kSweepMaxCols columns and 1 step)
    (void)H;
    const auto fits = [&](int r) { return int64_t(kSweepDepths) * ((int64_t(r) * W) | 1) <= kSweepPBuf; };
    if (W <= kSweepWaves * 6 && fits(8)) return 8;
    if (W <= kSweepWaves * kSweepMaxCols && fits(4)) return 4;
    return 0;
}

int bevpool_build_plan(const double *intrinsics, const double *extrinsics,
                       const int32_t *host_cells, const bevpool_geometry &g, hipStream_t stream,
                       bevpool_plan_s *plan) {
    const int64_t np64 = int64_t(g.n_cams) * g.n_depth * g.feat_h * g.feat_w;
    const int32_t np = int32_t(np64);
    const int32_t n_cells = g.nx * g.ny;
    const int32_t N = g.n_cams, D = g.n_depth, H = g.feat_h, W = g.feat_w;
    const int32_t HW = H * W;
    const int64_t n_combo = int64_t(N) * D * W;
    plan->n_points = np64;
    plan->n_cells = n_cells;
    plan->sweep_ok = (W <= kSweepWaves * kSweepMaxCols && bevpool_sweep_rows(W, H) > 0) ? 1 : 0;
    {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, plan->device) !=
                hipSuccess || cus < 1)
            cus = 256;
        plan->n_cus = cus;
    }

    int rc;
    if ((rc = dev_alloc(&plan->cell_of_point, size_t(np), "cell_of_point"))) return rc;
    if ((rc = dev_alloc(&plan->sorted_point, size_t(np), "sorted_point"))) return rc;
    if ((rc = dev_alloc(&plan->cell_start, size_t(n_cells) + 1, "cell_start"))) return rc;
    if ((rc = dev_alloc(&plan->column_table, size_t(n_combo), "column_table"))) return rc;
    if ((rc = dev_alloc(&plan->combo_cells, size_t(n_combo), "combo cells"))) return rc;

    // temporaries, carved from one arena that is freed on every exit path below
    const int64_t sort_cap = np64 > n_cells ? np64 : int64_t(n_cells);
    const int sort_tiles_cap = int((sort_cap + kSortTile - 1) / kSortTile);
    Arena arena;
    double *d_calib = nullptr;
    uint32_t *keys_a = nullptr, *keys_b = nullptr;
    int32_t *vals_a = nullptr, *vals_b = nullptr, *hist = nullptr, *small = nullptr;
    int32_t *scan_sums = nullptr;
    int32_t *flag_a = nullptr, *flag_b = nullptr, *flag_c = nullptr, *flag_x = nullptr;
    int32_t *combo_range = nullptr;
    int32_t *cell_generic = nullptr, *cell_ncombo = nullptr;
    int32_t *cell_key_min = nullptr, *cell_key_max = nullptr, *cell_w_min = nullptr,
            *cell_w_max = nullptr;
    int32_t *run_scan = nullptr, *run_begin = nullptr, *pos_of_cell = nullptr;
    auto cleanup = [&]() { (void)hipFree(arena.base); };

    // stable LSD radix sort of (keys, vals)[0, n) on the low `bits` bits; the
    // result ends in (keys, vals)
    auto radix_sort = [&](uint32_t *keys, int32_t *vals, int32_t n, int bits) -> int {
        if (n <= 0) return BEVPOOL_OK;
        const int tiles = int((int64_t(n) + kSortTile - 1) / kSortTile);
        const int passes = (bits + 7) / 8;
        uint32_t *kin = keys, *kout = keys == keys_a ? keys_b : keys_a;
        int32_t *vin = vals, *vout = vals == vals_b ? vals_a : vals_b;
        for (int pass = 0; pass < passes; ++pass) {
            const int shift = 8 * pass;
            hipLaunchKernelGGL(k_radix_hist, dim3(tiles), dim3(kBlock), 0, stream, kin, n, shift, hist);
            device_scan(hist, int64_t(tiles) * 256, small + 3, scan_sums, stream);
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
            // upper bounds of every temporary taken below: the kept points at
            // most the points, the generic cells at most the cells
            const size_t i4 = sizeof(int32_t);
            const size_t sort_b = Arena::piece(size_t(sort_cap) * i4);
            const size_t cells1_b = Arena::piece((size_t(n_cells) + 1) * i4);
            arena.cap = Arena::piece(size_t(g.n_cams) * 16 * sizeof(double)) + 4 * sort_b +
                        Arena::piece(size_t(sort_tiles_cap) * 256 * i4) + Arena::piece(16 * i4) +
                        Arena::piece(size_t(scan_sums_needed(sort_cap + 1)) * i4) +
                        10 * cells1_b +  // flags a/b/c, generic, ncombo, key min/max, w min/max, run_begin
                        Arena::piece((size_t(n_combo) + 1) * i4) +    // flag_x
                        Arena::piece(size_t(n_cells) * i4) +          // pos_of_cell
                        Arena::piece(size_t(n_combo) * i4) +          // combo_range
                        Arena::piece((size_t(np) + 1) * i4);          // run_scan
            if ((rc2 = dev_alloc(&arena.base, arena.cap, "plan temporaries"))) return rc2;
        }
        if (!host_cells && (rc2 = arena.take(&d_calib, size_t(g.n_cams) * 16, "calibration")))
            return rc2;
        if ((rc2 = arena.take(&keys_a, size_t(sort_cap), "sort keys"))) return rc2;
        if ((rc2 = arena.take(&keys_b, size_t(sort_cap), "sort keys"))) return rc2;
        if ((rc2 = arena.take(&vals_a, size_t(sort_cap), "sort values"))) return rc2;
        if ((rc2 = arena.take(&vals_b, size_t(sort_cap), "sort values"))) return rc2;
        if ((rc2 = arena.take(&hist, size_t(sort_tiles_cap) * 256, "radix histogram"))) return rc2;
        // [0..1] cell stats, [3] scan totals, [4..6] class counters, [8..13]
        // gathered counts
        if ((rc2 = arena.take(&small, 16, "plan counters"))) return rc2;
        // the longest scan is over sort_cap + 1 elements (radix histograms
        // are shorter)
        if ((rc2 = arena.take(&scan_sums, size_t(scan_sums_needed(sort_cap + 1)), "scan chunk sums")))
            return rc2;
        if ((rc2 = arena.take(&flag_a, size_t(n_cells) + 1, "flags"))) return rc2;
        if ((rc2 = arena.take(&flag_b, size_t(n_cells) + 1, "flags"))) return rc2;

        fill(small, 16, 0);
        if (host_cells) {
            // a stored association: the cell map as exported, checked by the caller
            BEVPOOL_HIP(hipMemcpyAsync(plan->cell_of_point, host_cells, sizeof(int32_t) * size_t(np),
                                       hipMemcpyHostToDevice, stream));
            hipLaunchKernelGGL(k_keys_from_cells, dim3(blocks_for(np)), dim3(kBlock), 0, stream,
                               plan->cell_of_point, np, n_cells, keys_a, plan->sorted_point);
        } else {
            BEVPOOL_HIP(hipMemcpyAsync(d_calib, intrinsics, sizeof(double) * 4 * g.n_cams,
                                       hipMemcpyHostToDevice, stream));
            BEVPOOL_HIP(hipMemcpyAsync(d_calib + 4 * g.n_cams, extrinsics,
                                       sizeof(double) * 12 * g.n_cams, hipMemcpyHostToDevice, stream));

            // Sec. III-B, precomputation: cell of every point, then the points
            // sorted by (cell, id) and the interval table.
            ProjectArgs pa;
            pa.intr = d_calib;
            pa.extr = d_calib + 4 * g.n_cams;
            pa.g = g;
            pa.div_w = make_fastdiv(uint32_t(W));
            pa.div_h = make_fastdiv(uint32_t(H));
            pa.div_d = make_fastdiv(uint32_t(D));
            pa.n_points = np;
            pa.n_cells = n_cells;
            pa.cell_of_point = plan->cell_of_point;
            pa.keys = keys_a;
            pa.vals = plan->sorted_point;
            hipLaunchKernelGGL(k_project, dim3(blocks_for(np)), dim3(kBlock), 0, stream, pa);
        }
        BEVPOOL_HIP(hipGetLastError());
        if ((rc2 = radix_sort(keys_a, plan->sorted_point, np, bits_for(n_cells)))) return rc2;
        hipLaunchKernelGGL(k_cell_start, dim3(blocks_for(int64_t(np) + 1)), dim3(kBlock), 0,
                           stream, keys_a, np, n_cells, plan->cell_start);
        hipLaunchKernelGGL(k_cell_stats, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, small);
        BEVPOOL_HIP(hipGetLastError());

        // combos, cell classes and the column table (the combo cells stay
        // with the plan: the backward pass reads them)
        if ((rc2 = arena.take(&combo_range, size_t(n_combo), "combo ranges"))) return rc2;
        if ((rc2 = arena.take(&cell_generic, size_t(n_cells), "cell classes"))) return rc2;
        if ((rc2 = arena.take(&cell_ncombo, size_t(n_cells), "cell combos"))) return rc2;
        if ((rc2 = arena.take(&cell_key_min, size_t(n_cells), "cell keys"))) return rc2;
        if ((rc2 = arena.take(&cell_key_max, size_t(n_cells), "cell keys"))) return rc2;
        if ((rc2 = arena.take(&cell_w_min, size_t(n_cells), "cell columns"))) return rc2;
        if ((rc2 = arena.take(&cell_w_max, size_t(n_cells), "cell columns"))) return rc2;
        fill(cell_generic, n_cells, 0);
        fill(cell_ncombo, n_cells, 0);
        fill(cell_key_min, n_cells, INT32_MAX);
        fill(cell_key_max, n_cells, -1);
        fill(cell_w_min, n_cells, INT32_MAX);
        fill(cell_w_max, n_cells, -1);
        ComboArgs ca;
        ca.cell_of_point = plan->cell_of_point;
        ca.N = N;
        ca.D = D;
        ca.H = H;
        ca.W = W;
        ca.allow_clean = H < kMaxFeatH ? 1 : 0;
        ca.sweep_ok = plan->sweep_ok;
        ca.combo_cell = plan->combo_cells;
        ca.combo_range = combo_range;
        ca.cell_generic = cell_generic;
        ca.cell_ncombo = cell_ncombo;
        ca.cell_key_min = cell_key_min;
        ca.cell_key_max = cell_key_max;
        ca.cell_w_min = cell_w_min;
        ca.cell_w_max = cell_w_max;
        hipLaunchKernelGGL(k_combo_walk, dim3(blocks_for(n_combo)), dim3(kBlock), 0, stream, ca);
        if ((rc2 = arena.take(&flag_c, size_t(n_cells) + 1, "flags"))) return rc2;
        if ((rc2 = arena.take(&flag_x, size_t(n_combo) + 1, "combo flags"))) return rc2;
        fill(flag_a, int64_t(n_cells) + 1, 0);
        fill(flag_b, int64_t(n_cells) + 1, 0);
        fill(flag_c, int64_t(n_cells) + 1, 0);
        hipLaunchKernelGGL(k_cell_class, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream, ca,
                           plan->cell_start, n_cells, flag_a, flag_b, flag_c, small + 4);
        hipLaunchKernelGGL(k_combo_table, dim3(blocks_for(n_combo)), dim3(kBlock), 0, stream, ca,
                           plan->column_table);
        device_scan(flag_a, int64_t(n_cells) + 1, small + 3, scan_sums, stream);   // run cells
        device_scan(flag_b, int64_t(n_cells) + 1, small + 3, scan_sums, stream);   // empty cells
        device_scan(flag_c, int64_t(n_cells) + 1, small + 3, scan_sums, stream);   // combo cells
        hipLaunchKernelGGL(k_cc_flags, dim3(blocks_for(n_combo + 1)), dim3(kBlock), 0, stream,
                           plan->combo_cells, n_combo, flag_c, flag_x);
        device_scan(flag_x, n_combo + 1, small + 3, scan_sums, stream);            // their combos
        BEVPOOL_HIP(hipGetLastError());
        hipLaunchKernelGGL(k_gather4, dim3(1), dim3(1), 0, stream, small + 8, flag_a + n_cells,
                           flag_b + n_cells, plan->cell_start + n_cells, small + 6);
        hipLaunchKernelGGL(k_gather4, dim3(1), dim3(1), 0, stream, small + 12, flag_c + n_cells,
                           flag_x + n_combo, small + 12, small + 12);
        BEVPOOL_HIP(hipGetLastError());
        int32_t h[16];
        BEVPOOL_HIP(hipMemcpyAsync(h, small, sizeof(h), hipMemcpyDeviceToHost, stream));
        BEVPOOL_HIP(hipStreamSynchronize(stream));
        const int32_t n_gen = h[8], n_empty = h[9], kept = h[10];
        const int32_t n_cc = h[12], n_cc_combos = h[13];
        plan->n_nonempty = h[0];
        plan->max_per_cell = h[1];
        plan->n_kept = kept;
        plan->n_column = h[4];
        plan->n_generic_heavy = h[5];
        plan->n_multi = h[11];
        plan->n_generic = n_gen + n_cc;
        plan->n_run_cells = n_gen;
        plan->n_combo_cells = n_cc;
        plan->n_cc_combos = n_cc_combos;
        plan->n_empty = n_empty;

        // combo cells: their combos grouped by cell (stable: combo order)
        if ((rc2 = dev_alloc(&plan->cc_hdr, size_t(n_cc), "combo-cell headers"))) return rc2;
        if ((rc2 = dev_alloc(&plan->cc_list, size_t(n_cc_combos), "combo-cell combos"))) return rc2;
        if (n_cc_combos > 0) {
            hipLaunchKernelGGL(k_cc_compact, dim3(blocks_for(n_combo)), dim3(kBlock), 0, stream,
                               plan->combo_cells, n_combo, flag_x, keys_a, vals_a);
            BEVPOOL_HIP(hipGetLastError());
            if ((rc2 = radix_sort(keys_a, vals_a, n_cc_combos, bits_for(n_cells)))) return rc2;
            hipLaunchKernelGGL(k_cc_list, dim3(blocks_for(n_cc_combos)), dim3(kBlock), 0, stream,
                               keys_a, vals_a, n_cc_combos, combo_range, flag_c, plan->cell_start,
                               plan->cc_list, plan->cc_hdr);
            BEVPOOL_HIP(hipGetLastError());
        }

        // cells without points, ascending
        if ((rc2 = dev_alloc(&plan->empty_cells, size_t(n_empty), "empty_cells"))) return rc2;
        hipLaunchKernelGGL(k_empty_list, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream, flag_b,
                           n_cells, plan->empty_cells);

        // generic cells by descending point count
        if ((rc2 = dev_alloc(&plan->generic_hdr, size_t(n_gen), "generic_hdr"))) return rc2;
        uint32_t *gen_key = keys_a;   // free again after the interval table
        int32_t *gen_cell = vals_a;
        hipLaunchKernelGGL(k_compact_generic, dim3(blocks_for(n_cells)), dim3(kBlock), 0, stream,
                           plan->cell_start, n_cells, flag_a, plan->max_per_cell, gen_key, gen_cell);
        BEVPOOL_HIP(hipGetLastError());
        if ((rc2 = radix_sort(gen_key, gen_cell, n_gen, bits_for(plan->max_per_cell)))) return rc2;

        // runs of the generic cells, in list order
        if ((rc2 = arena.take(&run_scan, size_t(kept) + 1, "run flags"))) return rc2;
        if ((rc2 = arena.take(&run_begin, size_t(n_gen) + 1, "run offsets"))) return rc2;
        if ((rc2 = arena.take(&pos_of_cell, size_t(n_cells), "cell positions"))) return rc2;
        fill(run_scan, int64_t(kept) + 1, 0);
        fill(run_begin, int64_t(n_gen) + 1, 0);
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
