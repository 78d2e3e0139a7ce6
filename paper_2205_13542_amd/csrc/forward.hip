// Per-frame BEV pooling: fused lift (depth probability x feature) and
// per-cell sum (BEVFusion, arXiv 2205.13542, Sec. III-B, first paragraph and
// "Interval Reduction"). The paper gives each cell one GPU thread that walks
// the cell's interval of sorted points. Here the work follows the camera
// geometry instead (see the partition in internal.h), in one launch whose
// workgroups take three kinds of work:
//
//   sweep          16 depth bins x 16 channels of one camera, over the
//                  camera's whole width. Each of the 16 waves owns a stretch
//                  of pixel columns. Per column it forms the column sums
//                  S[d][w][c] = sum_h P[d][h][w] F[h][w][c] on the matrix
//                  cores (v_mfma_f32_16x16x4f32: channels as M, depth bins as
//                  N, four pixel rows per step), with the depth probabilities
//                  staged in LDS by coalesced row loads and masked to each
//                  combo's kept rows. It then walks its columns in order,
//                  adding each depth bin's column sums into the current cell
//                  and storing the cell when its last column is reached. A
//                  cell that straddles two waves' stretches is finished
//                  through LDS. Every swept cell is stored once.
//   generic cells  cells seen by two cameras or by a tilted camera: their
//                  runs (consecutive depth bins of one pixel) are gathered by
//                  one wave, or by the whole workgroup for a cell with more
//                  than kGenHeavy points.
//   zero rows      cells without points, a share per workgroup, stored
//                  while the sweep's first loads are in flight.
//
// The same kernel takes the mean and the max (the "Interval Reduction"
// paragraph names both besides the sum). Mean: the sums divided by the
// cell's point count where a cell is stored. Max (MAXR): the column values
// are maxima over the rows, formed with vector instructions (a masked row
// carries a NaN probability, which fmaxf ignores), and cells combine their
// columns by max. Rows of the map are ldo floats apart (ldo >= C), so a call
// can fill one channel block of a wider map, e.g. one z slab.
//
// All reads and writes of P, F and the BEV map go through buffer resources
// of one frame each. An access that must not happen gets an offset past the
// end of its buffer: the hardware range check then returns 0 for a load and
// drops a store. Every output row gets its value from one plain store, and
// every sum runs in an order fixed by the plan, so results are
// deterministic.
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include <hip/hip_ext.h>

#include "device.h"
#include "internal.h"

namespace bevpool {
namespace {

typedef float f4v __attribute__((ext_vector_type(4)));

struct FwdArgs {
    const char *P, *F;
    float *out;
    const int2 *table;
    const int4 *gen_hdr;
    const int4 *gen_runs;
    const int4 *cc_hdr;                 // combo cells: headers, then their combos
    const int2 *cc_list;
    const int32_t *empty_cells;
    const int32_t *cell_start;          // interval table: point counts of the cells
    int32_t N, D, H, W, HW, C;
    int32_t n_cells, ldo, mean, vec_out;
    uint32_t p_bytes, f_bytes, o_bytes, run_bytes;   // per frame (runs: whole table)
    uint32_t table_bytes, empty_bytes;  // column table, empty-cell list
    uint32_t cc_bytes;                  // combo-cell combo list
    int32_t n_cc;                       // combo cells
    FastDiv div_w, div_d;               // division by W, by D (combo ids)
    // sweep workgroups (camera, depth tile, channel tile)
    int32_t n_sweep, n_dt, n_ct;
    int32_t rows, n_chunks;             // staged rows per chunk (4 or 8), chunks
    int32_t ds;                         // LDS stride of a depth bin's staged probabilities
    int32_t waves;                      // waves that own columns: min(kSweepWaves, W)
    // generic cells, zero rows
    int32_t n_heavy, n_light;
    int32_t slice_c, n_slices;
    int32_t n_empty, zero_vec, zero_units, row_units;
    FastDiv div_units;
};

// The buffers of frame b: depth probabilities, features, BEV map.
struct Frame {
    Rsrc P, F, O;
    __device__ __forceinline__ Frame(const FwdArgs &a, int b)
        : P(make_rsrc(a.P + int64_t(b) * a.p_bytes, a.p_bytes)),
          F(make_rsrc(a.F + int64_t(b) * a.f_bytes, a.f_bytes)),
          O(make_rsrc(reinterpret_cast<const char *>(a.out) + int64_t(b) * a.o_bytes, a.o_bytes)) {}
};

// LDS of a workgroup. The staged probabilities of the sweep (two buffers)
// also hold the lane-group partials of a heavy generic cell afterwards.
constexpr int kInfoE = 1, kInfoClose = 2, kInfoX = 4;
struct SweepLds {
    float p[2][kSweepPBuf];
    f4v e[kSweepWaves][kWaveSize];      // partial of the cell open at a wave's first column
    f4v x[kSweepWaves][kWaveSize];      // partial of the cell open past a wave's last column
    int info[kSweepWaves][kSweepDepths];
    int ecell[kSweepWaves][kSweepDepths];
    int ecnt[kSweepWaves][kSweepDepths];   // point counts of those partials
    int xcnt[kSweepWaves][kSweepDepths];
    int cell[kSweepWaves][kSweepDepths][kSweepMaxCols];   // cells of a wave's columns
};

// Largest staged probabilities per lane and chunk (16 depth bins x rows x W
// values fill at most one buffer, one wave per depth bin).
constexpr int kStageMax = kSweepPBuf / kSweepBlock;
static_assert(kSweepPBuf % kSweepBlock == 0, "whole staging rounds");
// Zero-row units a thread stores per batch.
constexpr int kZeroBatch = 8;
// Light generic cells a wave of a workgroup without a sweep takes, at most,
// before the sweep workgroups share the rest.
constexpr int kGenPerWave = 4;

// LDS row stride of a lane group's partial sums for a heavy generic cell.
template <int NCH>
constexpr int slot_stride() { return 16 * NCH + ((NCH % 2 == 0) ? 16 : 0); }

__device__ __forceinline__ f4v f4_init(bool maxr) {
    const float v = maxr ? -INFINITY : 0.f;
    return (f4v){v, v, v, v};
}

template <bool MAXR>
__device__ __forceinline__ f4v f4_join(f4v s, f4v v) {
    if constexpr (MAXR)
        return (f4v){fmaxf(s[0], v[0]), fmaxf(s[1], v[1]), fmaxf(s[2], v[2]), fmaxf(s[3], v[3])};
    else
        return s + v;
}

// Store channels c0 + 4q .. c0 + 4q + 3 of a swept cell's row when `store`
// holds (a lane that does not store gets offsets past the buffer); the mean
// divides by the cell's point count first.
__device__ __forceinline__ void store_cell(const FwdArgs &a, Rsrc out, bool store, int cell, int cq,
                                           f4v v, bool mean, int cnt) {
    if (mean) v = v / float(cnt > 0 ? cnt : 1);
    const uint32_t row = uint32_t(cell) * uint32_t(a.ldo);
    if (a.vec_out && cq + 4 <= a.C) {
        __builtin_amdgcn_raw_buffer_store_b128(
            (__attribute__((ext_vector_type(4))) uint32_t){__float_as_uint(v[0]), __float_as_uint(v[1]),
                                                           __float_as_uint(v[2]), __float_as_uint(v[3])},
            out, int(store ? (row + uint32_t(cq)) * 4u : kOff), 0, 0);
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            store_f32(out, store && cq + k < a.C ? (row + uint32_t(cq + k)) * 4u : kOff, v[k]);
    }
}

// Workgroup g's share of the empty rows, as units of 16 bytes (or 4 bytes
// when rows are not 16-byte aligned): unit f is unit f % U of row f / U.
// Rows of consecutive cells are adjacent, so runs of empty cells become
// contiguous stores. zero_cells loads the cell ids of one batch, zero_store
// stores it; a thread's units of a batch are f = t + k * kSweepBlock.
struct ZeroBatch {
    int cell[kZeroBatch];
};
__device__ __forceinline__ void zero_range(const FwdArgs &a, int g, int G, int &e0, int &total) {
    const int z0 = int(int64_t(a.n_empty) * g / G), z1 = int(int64_t(a.n_empty) * (g + 1) / G);
    e0 = z0;
    total = (z1 - z0) * a.zero_units;
}
__device__ __forceinline__ void zero_cells(const FwdArgs &a, int e0, int total, int f0, ZeroBatch &zb) {
    const Rsrc list = make_rsrc(a.empty_cells, a.empty_bytes);
#pragma unroll
    for (int k = 0; k < kZeroBatch; ++k) {
        const int f = f0 + k * kSweepBlock + int(threadIdx.x);
        const uint32_t off = uint32_t(e0 + int(fdiv(uint32_t(f), a.div_units))) * 4u;
        zb.cell[k] = int(__builtin_amdgcn_raw_buffer_load_b32(list, int(f < total ? off : kOff), 0, 0));
    }
}
__device__ __forceinline__ void zero_store(const FwdArgs &a, Rsrc out, int total, int f0,
                                           const ZeroBatch &zb, int part = 0, int every = 1) {
#pragma unroll
    for (int k = 0; k < kZeroBatch; ++k) {
        if (k % every != part) continue;
        const int f = f0 + k * kSweepBlock + int(threadIdx.x);
        const int r = int(fdiv(uint32_t(f), a.div_units));
        const uint32_t u = uint32_t(f - r * a.zero_units);
        const bool ok = f < total;
        if (a.zero_vec) {
            __builtin_amdgcn_raw_buffer_store_b128(
                (__attribute__((ext_vector_type(4))) uint32_t){0u, 0u, 0u, 0u}, out,
                int(ok ? (uint32_t(zb.cell[k]) * uint32_t(a.row_units) + u) * 16u : kOff), 0, 0);
        } else {
            store_f32(out, ok ? (uint32_t(zb.cell[k]) * uint32_t(a.row_units) + u) * 4u : kOff, 0.f);
        }
    }
}

// The sweep of workgroup (camera n, depth tile, channel tile) sg, NC columns
// per wave at most and RK matrix-core steps (of 4 rows) per staged chunk at
// most. zb holds the zero-row batch whose cell ids were loaded before the
// sweep's first loads; it is stored once those are issued.
template <int DT, bool MAXR, int NC, int RK>
__device__ void sweep(const FwdArgs &a, const Frame &fr, int sg, SweepLds &s, const ZeroBatch &zb,
                      int ztotal) {
    constexpr uint32_t ES = Elem<DT>::kBytes;
    constexpr int R = 4 * RK;   // staged rows per chunk
    const int ct = sg % a.n_ct, t2 = sg / a.n_ct;
    const int dtile = t2 % a.n_dt, n = t2 / a.n_dt;
    const int d0 = dtile * kSweepDepths, c0 = ct * kSweepChannels;
    // wave-uniform values in scalar registers (readfirstlane), so that the
    // masks built from them stay selects rather than branches
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int q = lane >> 4, j = lane & 15;
    const int W = a.W, H = a.H;
    const int nwv = a.waves;
    const int wb = __builtin_amdgcn_readfirstlane(wave < nwv ? int(int64_t(wave) * W / nwv) : W);
    const int nc = __builtin_amdgcn_readfirstlane(wave < nwv ? int(int64_t(wave + 1) * W / nwv) - wb : 0);
    const int d = d0 + j;   // this lane's depth bin (matrix-core column)

    // The column-table entries of depth bin d at this wave's columns (a
    // column past the wave's stretch reads as inactive: out-of-range loads
    // return zeros). The row range becomes, for this lane's rows
    // q, q + 4, ..., the bounds lo - q <= r0 + 4 * step < hi - q on the
    // uniform row index r0 + 4 * step; cells go to LDS for the walk.
    const Rsrc tab = make_rsrc(a.table, a.table_bytes);
    const uint32_t trow = uint32_t((n * W + wb) * a.D + d) * 8u;   // table [N][W][D]
    const uint32_t tcol = uint32_t(a.D) * 8u;
    int ey[NC], rlo[NC], rspan[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        const auto e = __builtin_amdgcn_raw_buffer_load_b64(
            tab, int(((i < nc) & (d < a.D)) ? trow + uint32_t(i) * tcol : kOff), 0, 0);
        ey[i] = int(e[0]) >= 0 ? int(e[1]) : 0;
        s.cell[wave][j][i] = int(e[0]);   // read back by the walk (the 4 lanes of a depth bin agree)
        const int lo = ey[i] & 0x7FFF, hi = (ey[i] >> 15) & 0x7FFF;
        rlo[i] = lo - q;
        rspan[i] = hi - lo;   // 0 for an inactive column: every row masked
    }
    if (q == 0) s.info[wave][j] = 0;

    // Staging of chunk c (rows c * R .. c * R + R - 1): for each of the 16
    // depth bins those rows are R * W consecutive values of P, kept in LDS in
    // the same order, depth bins ds values apart (ds odd: the 64 lanes of a
    // matrix-core step, 16 depth bins x 4 rows, then meet distinct banks when
    // W is 8 or 24 modulo 32). Wave dd stages depth bin d0 + dd, its lane l
    // the offsets l, l + 64, ... of the chunk. The loads need no mask: past
    // the chunk they read the following rows (or zeros past the buffer),
    // which only the LDS store leaves out, and rows past H are masked where
    // they are used (no combo keeps them).
    static_assert(kSweepWaves == kSweepDepths, "one staging wave per depth bin");
    const int rw = R * W;
    const uint32_t pdepth = d0 + wave < a.D ? uint32_t((n * a.D + d0 + wave) * H) * uint32_t(W) * ES : kOff;
    const uint32_t plane = uint32_t(lane) * ES;
    float pv[kStageMax];
    auto stage_load = [&](int c) {
        const uint32_t sbase = pdepth + uint32_t(c * rw) * ES;   // uniform
#pragma unroll
        for (int k = 0; k < kStageMax; ++k)
            pv[k] = Elem<DT>::load(fr.P, sbase + plane + uint32_t(k * kWaveSize) * ES);
    };
    auto stage_store = [&](int buf) {
        float *dst = &s.p[buf][wave * a.ds + lane];
#pragma unroll
        for (int k = 0; k < kStageMax; ++k) {
            if ((k + 1) * kWaveSize <= rw) dst[k * kWaveSize] = pv[k];
            else if (lane + k * kWaveSize < rw) dst[k * kWaveSize] = pv[k];
        }
    };
    // LDS word of depth bin j, chunk row 4 * st + q, wave column 0
    const int pl_base = j * a.ds + q * W + wb;

    f4v acc[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) acc[i] = f4_init(MAXR);
    // the k-th chunk this workgroup processes: workgroups that read the same
    // lines (the depth tiles of one camera share its feature rows, the
    // channel tiles its probabilities) start at different chunks, so that
    // they do not request one line at the same moment
    const int cstart = (dtile + ct) % a.n_chunks;
    auto chunk_at = [&](int k) { const int c = cstart + k; return c < a.n_chunks ? c : c - a.n_chunks; };

    if constexpr (!MAXR) {
        // matrix-core operand A: lane (k = q, m = j) holds F[n][r][w][c0 + j]
        // for row r = r0 + 4 * step + q; the column part of the offset is
        // per lane and fixed, the row part uniform
        uint32_t fcol[NC];
        const bool cok = c0 + j < a.C;
#pragma unroll
        for (int i = 0; i < NC; ++i)
            fcol[i] = ((i < nc) & cok)
                          ? ((uint32_t(n * H + q) * uint32_t(W) + uint32_t(wb + i)) * uint32_t(a.C) +
                             uint32_t(c0 + j)) * ES
                          : kOff;
        const uint32_t frow = uint32_t(W) * uint32_t(a.C) * ES;   // one pixel row
        auto f_load = [&](float (&fa)[NC][RK], int c) {
#pragma unroll
            for (int st = 0; st < RK; ++st) {
                const uint32_t roff = uint32_t(c * R + 4 * st) * frow;   // uniform
#pragma unroll
                for (int i = 0; i < NC; ++i) fa[i][st] = Elem<DT>::load(fr.F, fcol[i] + roff);
            }
        };
        // One chunk: issue the next chunk's loads, read this chunk's
        // probabilities from LDS (all before the first product), run the
        // products, then store the next chunk's probabilities. The buffer
        // index is a constant of each instance, so both feature buffers stay
        // in fixed registers.
        float fa0[NC][RK], fa1[NC][RK];
        auto chunk = [&](auto buf_c, int k, float (&cur)[NC][RK], float (&nxt)[NC][RK]) {
            constexpr int buf = decltype(buf_c)::value;
            const bool more = k + 1 < a.n_chunks;
            const int c = chunk_at(k);
            if (more) {
                stage_load(chunk_at(k + 1));
                f_load(nxt, chunk_at(k + 1));
            }
            // a slice of this workgroup's empty rows, stored while the
            // chunk computes (its cell ids were loaded first of all)
            zero_store(a, fr.O, ztotal, 0, zb, k, a.n_chunks);
            float pb[NC][RK];
#pragma unroll
            for (int st = 0; st < RK; ++st) {
                const float *src = &s.p[buf][pl_base + 4 * st * W];
                const int r = c * R + 4 * st;   // uniform row index of this step
#pragma unroll
                for (int i = 0; i < NC; ++i) {
                    const float pval = src[i];
                    pb[i][st] = uint32_t(r - rlo[i]) < uint32_t(rspan[i]) ? pval : 0.f;
                }
            }
            // every wave runs NC columns: past its stretch both operands are 0
#pragma unroll
            for (int st = 0; st < RK; ++st)
#pragma unroll
                for (int i = 0; i < NC; ++i)
                    acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(cur[i][st], pb[i][st], acc[i], 0, 0, 0);
            if (more) stage_store(buf ^ 1);
            __syncthreads();
        };
        stage_load(cstart);
        f_load(fa0, cstart);
        stage_store(0);
        __syncthreads();
        for (int k = 0; k < a.n_chunks; k += 2) {
            chunk(std::integral_constant<int, 0>(), k, fa0, fa1);
            if (k + 1 < a.n_chunks) chunk(std::integral_constant<int, 1>(), k + 1, fa1, fa0);
        }
    } else {
        // vector maxima: lane (q, j) holds channels c0 + 4q .. + 3 of depth
        // bin d; per row, max(acc, p * f), a masked row carrying NaN
        stage_load(cstart);
        stage_store(0);
        __syncthreads();
        const int cq = c0 + 4 * q;
        for (int k = 0; k < a.n_chunks; ++k) {
            const int buf = k & 1;
            const bool more = k + 1 < a.n_chunks;
            const int c = chunk_at(k);
            if (more) stage_load(chunk_at(k + 1));
            zero_store(a, fr.O, ztotal, 0, zb, k, a.n_chunks);
            const int r0 = c * R;
#pragma unroll
            for (int i = 0; i < NC; ++i) {
                if (i < nc) {
                    for (int rr = 0; rr < R; ++rr) {
                        const int r = r0 + rr;
                        const float pv_ = s.p[buf][j * a.ds + rr * W + wb + i];
                        const uint32_t y = uint32_t(ey[i]);
                        const uint32_t lo = y & 0x7FFFu, hi = (y >> 15) & 0x7FFFu;
                        const float p = uint32_t(r) - lo < hi - lo ? pv_ : __builtin_nanf("");
                        const uint32_t fo = (uint32_t(n * H + r) * uint32_t(W) + uint32_t(wb + i)) * uint32_t(a.C);
#pragma unroll
                        for (int kk = 0; kk < 4; ++kk) {
                            const float f = Elem<DT>::load(fr.F, ((r < H) & (cq + kk < a.C)) ? (fo + uint32_t(cq + kk)) * ES : kOff);
                            acc[i][kk] = fmaxf(acc[i][kk], p * f);
                        }
                    }
                }
            }
            if (more) stage_store(buf ^ 1);
            __syncthreads();
        }
    }

    // Walk this wave's columns in order: lane (q, j) holds channels
    // c0 + 4q .. c0 + 4q + 3 of depth bin d0 + j for every column. A cell's
    // columns are consecutive; the cell is stored at its last column, unless
    // it began before this wave's first column (its partial goes to e) or
    // runs past the last one (its partial goes to x). A cell's point count
    // (for the mean) is the sum of its columns' kept rows.
    const bool mean = !MAXR && a.mean != 0;
    const int cq = c0 + 4 * q;
    f4v S = f4_init(MAXR);
    int cnt = 0;
    bool open = false, pending = false;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        const uint32_t y = uint32_t(ey[i]);
        const bool act = rspan[i] > 0;   // false past the wave's stretch
        if (i == 0) open = act && !(y & kColFirst);
        if (act) {
            S = f4_join<MAXR>(S, acc[i]);
            cnt += rspan[i];
        }
        const bool last = act && (y & kColLast);
        // a cell that began before this wave and ends here: its partial for
        // the combine; any other cell ending here is stored
        const bool to_e = last && open;
        if (to_e) {
            s.e[wave][lane] = S;
            if (q == 0) {
                s.info[wave][j] = kInfoE | kInfoClose;
                s.ecell[wave][j] = s.cell[wave][j][i];
                s.ecnt[wave][j] = cnt;
            }
        }
        store_cell(a, fr.O, last && !open, s.cell[wave][j][i], cq, S, mean, cnt);
        if (last) {
            S = f4_init(MAXR);
            cnt = 0;
            open = false;
        }
        if (i < nc) pending = act && !last;
    }
    if (pending) {
        if (open) {
            s.e[wave][lane] = S;
            if (q == 0) {
                s.info[wave][j] = kInfoE;
                s.ecnt[wave][j] = cnt;
            }
        } else {
            s.x[wave][lane] = S;
            if (q == 0) {
                s.info[wave][j] |= kInfoX;
                s.xcnt[wave][j] = cnt;
            }
        }
    }
    __syncthreads();
    // Cells that straddle waves, finished by the wave where they end: its
    // partial, the partials of the waves they span whole, and the partial of
    // the wave where they began, added from left to right.
    {
        const int inf = s.info[wave][j];
        if ((inf & kInfoE) && (inf & kInfoClose)) {
            int k0 = wave - 1;
            while (k0 > 0 && (s.info[k0][j] & (kInfoE | kInfoClose)) == kInfoE) --k0;
            // wave k0 holds the cell's first partial (x), waves k0+1 .. wave the rest (e)
            f4v T = s.x[k0][lane];
            int tc = s.xcnt[k0][j];
            for (int k = k0 + 1; k <= wave; ++k) {
                T = f4_join<MAXR>(T, s.e[k][lane]);
                tc += s.ecnt[k][j];
            }
            store_cell(a, fr.O, true, s.ecell[wave][j], cq, T, mean, tc);
        }
    }
}

// A generic cell's runs in chunks of 64: lane i loads run i of the chunk and
// sums its depth probabilities; then the four lane groups take the runs
// round-robin, four at a time, each run costing one feature row. A group's
// runs are added in a fixed order. With MAXR a run's points share one
// feature row f, so their largest product per channel is f times the run's
// largest probability where f >= 0 and f times its smallest otherwise; a
// run past the chunk carries NaN probabilities, which fmaxf ignores.
template <int DT, int NCH, bool VEC, bool MAXR>
__device__ __forceinline__ void generic_runs(float (&acc)[NCH], const FwdArgs &a, const Frame &fr,
                                             int4 hdr, int c0, int first_chunk, int chunk_step) {
    constexpr uint32_t ES = Elem<DT>::kBytes;
    const int lane = threadIdx.x & 63;
    const int grp = lane >> 4;
    const Rsrc runs = make_rsrc(a.gen_runs, a.run_bytes);
    for (int ch = first_chunk; ch * 64 < hdr.z; ch += chunk_step) {
        const int nr = min(64, hdr.z - ch * 64);
        const uint32_t roff = lane < nr ? uint32_t(hdr.y + ch * 64 + lane) * 16u : kOff;
        const auto rv = __builtin_amdgcn_raw_buffer_load_b128(runs, int(roff), 0, 0);
        const int p0 = int(rv[0]), pix = int(rv[1]), len = int(rv[2]);
        float ps = 0.f, pmin = INFINITY;   // sum (max with MAXR) and min of the run's probabilities
        if constexpr (MAXR) ps = -INFINITY;
        for (int qd = 0; qd < len; ++qd) {
            const float pq = Elem<DT>::load(fr.P, uint32_t(p0 + qd * a.HW) * ES);
            if constexpr (MAXR) {
                ps = fmaxf(ps, pq);
                pmin = fminf(pmin, pq);
            } else {
                ps += pq;
            }
        }
        for (int i0 = 0; i0 < nr; i0 += 16) {
            float pr[4], pm[4];
            Row<NCH> f[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + 4 * u + grp;
                pr[u] = __shfl(ps, i & 63);
                pm[u] = __shfl(pmin, i & 63);
                if (MAXR && i >= nr) pr[u] = pm[u] = __builtin_nanf("");
                const int px = __shfl(pix, i & 63);
                load_row<DT, NCH, VEC>(f[u], fr.F,
                                       i < nr ? (uint32_t(px) * uint32_t(a.C) + uint32_t(c0)) * ES : kOff);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int k = 0; k < NCH; ++k) {
                    if constexpr (MAXR)
                        acc[k] = fmaxf(acc[k], (f[u].v[k] >= 0.f ? pr[u] : pm[u]) * f[u].v[k]);
                    else
                        acc[k] = __builtin_fmaf(pr[u], f[u].v[k], acc[k]);
                }
        }
    }
}

// Mean: a generic cell's total divided by its point count.
template <int NCH>
__device__ __forceinline__ void divide_by_count(float (&v)[NCH], const FwdArgs &a, int cell) {
    const float cnt = float(a.cell_start[cell + 1] - a.cell_start[cell]);
#pragma unroll
    for (int q = 0; q < NCH; ++q) v[q] = v[q] / cnt;
}

template <int DT, int NCH, bool VEC, bool MAXR>
__device__ void light_generic(const FwdArgs &a, const Frame &fr, int k, int c0, int cn) {
    const int lane = threadIdx.x & 63;
    const int j = lane & 15, grp = lane >> 4;
    const int4 hdr = a.gen_hdr[a.n_heavy + k];
    float acc[NCH];
#pragma unroll
    for (int q = 0; q < NCH; ++q) acc[q] = MAXR ? -INFINITY : 0.f;
    generic_runs<DT, NCH, VEC, MAXR>(acc, a, fr, hdr, c0, 0, 1);
    // (g0 + g1) + (g2 + g3), the same in every lane of the wave
#pragma unroll
    for (int q = 0; q < NCH; ++q) {
        if constexpr (MAXR) {
            const float s = fmaxf(acc[q], __shfl_xor(acc[q], 16));
            acc[q] = fmaxf(s, __shfl_xor(s, 32));
        } else {
            const float s = acc[q] + __shfl_xor(acc[q], 16);
            acc[q] = s + __shfl_xor(s, 32);
        }
    }
    if (!MAXR && a.mean) divide_by_count<NCH>(acc, a, hdr.x);
    store_row<NCH, VEC>(fr.O, grp == 0 ? (uint32_t(hdr.x) * uint32_t(a.ldo) + uint32_t(c0)) * 4u : kOff,
                        acc, j + 16 * (NCH - 1) < cn);
}

// A combo cell (a generic cell whose points all lie in clean combos, e.g. a
// cell that two cameras see), one wave: its combos in order, each one a
// pixel column of one depth bin with a range of kept rows. The four lane
// groups take the rows q, q + 4, ... of a combo, all of them loaded at once,
// and are added at the end in a fixed order.
template <int DT, int NCH, bool VEC, bool MAXR>
__device__ void combo_cell(const FwdArgs &a, const Frame &fr, int k, int c0, int cn) {
    constexpr uint32_t ES = Elem<DT>::kBytes;
    constexpr int kRows = 8;   // rows a lane group loads per pass
    const int lane = threadIdx.x & 63;
    const int q = lane >> 4, j = lane & 15;
    const int4 hdr = a.cc_hdr[k];
    const Rsrc lst = make_rsrc(a.cc_list, a.cc_bytes);
    const int W = a.W, H = a.H;
    float acc[NCH];
#pragma unroll
    for (int t = 0; t < NCH; ++t) acc[t] = MAXR ? -INFINITY : 0.f;
    for (int e0 = 0; e0 < hdr.z; e0 += kWaveSize) {
        const int ne = min(kWaveSize, hdr.z - e0);
        const auto ent = __builtin_amdgcn_raw_buffer_load_b64(
            lst, int(lane < ne ? uint32_t(hdr.y + e0 + lane) * 8u : kOff), 0, 0);
        for (int e = 0; e < ne; ++e) {
            const uint32_t X = uint32_t(__shfl(int(ent[0]), e));
            const uint32_t rg = uint32_t(__shfl(int(ent[1]), e));
            const uint32_t nd = fdiv(X, a.div_w);
            const uint32_t w = X - nd * uint32_t(W);
            const uint32_t n = fdiv(nd, a.div_d);
            const int lo = int(rg & 0x7FFFu), hi = int((rg >> 15) & 0x7FFFu);
            const uint32_t pcol = nd * uint32_t(H) * uint32_t(W) + w;                 // P[n][d][0][w]
            const uint32_t fcol = (n * uint32_t(H) * uint32_t(W) + w) * uint32_t(a.C) + uint32_t(c0);
            for (int hb = lo - (lo & 3); hb < hi; hb += 4 * kRows) {
                float p[kRows];
                Row<NCH> f[kRows];
#pragma unroll
                for (int t = 0; t < kRows; ++t) {
                    const int h = hb + q + 4 * t;
                    const bool ok = (h >= lo) & (h < hi);
                    p[t] = Elem<DT>::load(fr.P, ok ? (pcol + uint32_t(h) * uint32_t(W)) * ES : kOff);
                    if (MAXR && !ok) p[t] = __builtin_nanf("");
                    load_row<DT, NCH, VEC>(f[t], fr.F,
                                           ok ? (fcol + uint32_t(h) * uint32_t(W) * uint32_t(a.C)) * ES : kOff);
                }
#pragma unroll
                for (int t = 0; t < kRows; ++t)
#pragma unroll
                    for (int kk = 0; kk < NCH; ++kk) {
                        if constexpr (MAXR)
                            acc[kk] = fmaxf(acc[kk], p[t] * f[t].v[kk]);
                        else
                            acc[kk] = __builtin_fmaf(p[t], f[t].v[kk], acc[kk]);
                    }
            }
        }
    }
    // (g0 + g1) + (g2 + g3), the same in every lane of the wave
#pragma unroll
    for (int t = 0; t < NCH; ++t) {
        if constexpr (MAXR) {
            const float s = fmaxf(acc[t], __shfl_xor(acc[t], 16));
            acc[t] = fmaxf(s, __shfl_xor(s, 32));
        } else {
            const float s = acc[t] + __shfl_xor(acc[t], 16);
            acc[t] = s + __shfl_xor(s, 32);
        }
    }
    if (!MAXR && a.mean) {
#pragma unroll
        for (int t = 0; t < NCH; ++t) acc[t] = acc[t] / float(hdr.w);
    }
    store_row<NCH, VEC>(fr.O, q == 0 ? (uint32_t(hdr.x) * uint32_t(a.ldo) + uint32_t(c0)) * 4u : kOff,
                        acc, j + 16 * (NCH - 1) < cn);
}

// A heavy generic cell: the workgroup's waves take its run chunks in turn;
// the 4 * kSweepWaves lane-group partials are added in a fixed order.
template <int DT, int NCH, bool VEC, bool MAXR>
__device__ void heavy_generic(const FwdArgs &a, const Frame &fr, int k, int c0, int cn,
                              float *s_part) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15;
    const int wl = wave * 4 + (lane >> 4);
    constexpr int SS = slot_stride<NCH>();
    const int4 hdr = a.gen_hdr[k];
    float acc[NCH];
#pragma unroll
    for (int q = 0; q < NCH; ++q) acc[q] = MAXR ? -INFINITY : 0.f;
    generic_runs<DT, NCH, VEC, MAXR>(acc, a, fr, hdr, c0, wave, kSweepWaves);
#pragma unroll
    for (int q = 0; q < NCH; ++q) s_part[wl * SS + j + 16 * q] = acc[q];
    __syncthreads();
    if (wl == 0) {
        float sum[NCH];
#pragma unroll
        for (int q = 0; q < NCH; ++q) sum[q] = MAXR ? -INFINITY : 0.f;
        for (int g = 0; g < 4 * kSweepWaves; ++g)
#pragma unroll
            for (int q = 0; q < NCH; ++q) {
                if constexpr (MAXR)
                    sum[q] = fmaxf(sum[q], s_part[g * SS + j + 16 * q]);
                else
                    sum[q] += s_part[g * SS + j + 16 * q];
            }
        if (!MAXR && a.mean) divide_by_count<NCH>(sum, a, hdr.x);
        store_row<NCH, VEC>(fr.O, (uint32_t(hdr.x) * uint32_t(a.ldo) + uint32_t(c0)) * 4u, sum,
                            j + 16 * (NCH - 1) < cn);
    }
    __syncthreads();
}
static_assert(4 * kSweepWaves * slot_stride<8>() <= 2 * kSweepPBuf, "heavy partials fit the staging LDS");

// Sweep groups are placed so that consecutive ones (the channel tiles of
// one camera and depth tile, which stage the same probabilities) share an
// XCD's L2 (xcd_cu_remap in device.h).
template <int DT, int NCH, bool VEC, bool MAXR, int NC>
__global__ __launch_bounds__(kSweepBlock) void k_forward(FwdArgs a) {
    __shared__ SweepLds s;
    const int G = int(gridDim.x), b = blockIdx.y;
    const int g = int(blockIdx.x);
    const Frame fr(a, b);

    // this workgroup's share of the empty rows: the first batch's cell ids
    // are loaded before anything else, so that storing them waits for
    // nothing that the sweep issues
    int ze0, ztotal;
    zero_range(a, g, G, ze0, ztotal);
    ZeroBatch zb;
    zero_cells(a, ze0, ztotal, 0, zb);

    const int sg = xcd_cu_remap<1>(g, G);
    const int Gs = a.n_sweep, Gn = G - Gs;   // sweep and other workgroups
    const bool swp = sg < Gs;
    const int wave = threadIdx.x >> 6;

    // Generic cells, channel slice by slice: wave items (combo cells, then
    // light run cells) and workgroup items (heavy run cells). The workgroups
    // without a sweep take them first, from the start of the launch beside
    // the sweeps: up to kGenPerWave wave items a wave and every heavy cell;
    // the sweep workgroups take the rest after their sweep.
    const int n_items = a.n_cc + a.n_light;
    const int ln = Gn > 0 ? min(n_items, Gn * kSweepWaves * kGenPerWave) : 0;
    auto item = [&](int it, int c0, int cn) {
        if (it < a.n_cc) combo_cell<DT, NCH, VEC, MAXR>(a, fr, it, c0, cn);
        else light_generic<DT, NCH, VEC, MAXR>(a, fr, it - a.n_cc, c0, cn);
    };
    auto generic = [&](bool first) {
        for (int sl = 0; sl < a.n_slices; ++sl) {
            const int c0 = sl * a.slice_c;
            const int cn = min(a.slice_c, a.C - c0);
            if (first) {
                for (int h = sg - Gs; h < a.n_heavy; h += Gn)
                    heavy_generic<DT, NCH, VEC, MAXR>(a, fr, h, c0, cn, &s.p[0][0]);
                for (int it = (sg - Gs) * kSweepWaves + wave; it < ln; it += Gn * kSweepWaves)
                    item(it, c0, cn);
            } else {
                if (Gn == 0)
                    for (int h = sg; h < a.n_heavy; h += Gs)
                        heavy_generic<DT, NCH, VEC, MAXR>(a, fr, h, c0, cn, &s.p[0][0]);
                for (int it = ln + sg * kSweepWaves + wave; it < n_items; it += Gs * kSweepWaves)
                    item(it, c0, cn);
            }
        }
    };

    if (swp) {
        sweep<DT, MAXR, NC, (NC > 6 ? 1 : 2)>(a, fr, sg, s, zb, ztotal);   // rows = 4 * RK
    } else {
        generic(true);
        zero_store(a, fr.O, ztotal, 0, zb);
    }
    for (int f0 = kZeroBatch * kSweepBlock; f0 < ztotal; f0 += kZeroBatch * kSweepBlock) {
        zero_cells(a, ze0, ztotal, f0, zb);
        zero_store(a, fr.O, ztotal, f0, zb);
    }
    if (swp) generic(false);
}

template <int DT, bool MAXR, int NC>
void launch_nch(const FwdArgs &a, dim3 grid, int nch, bool vec, hipStream_t s, hipEvent_t e0,
                hipEvent_t e1) {
    const dim3 block(kSweepBlock);
    switch (nch) {
        case 1: hipExtLaunchKernelGGL((k_forward<DT, 1, false, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a); break;
        case 2: hipExtLaunchKernelGGL((k_forward<DT, 2, false, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a); break;
        case 3: hipExtLaunchKernelGGL((k_forward<DT, 3, false, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a); break;
        case 4:
            if (vec) hipExtLaunchKernelGGL((k_forward<DT, 4, true, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a);
            else hipExtLaunchKernelGGL((k_forward<DT, 4, false, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a);
            break;
        case 5:
            if (vec) hipExtLaunchKernelGGL((k_forward<DT, 5, true, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a);
            else hipExtLaunchKernelGGL((k_forward<DT, 5, false, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a);
            break;
        case 6: hipExtLaunchKernelGGL((k_forward<DT, 6, false, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a); break;
        case 7: hipExtLaunchKernelGGL((k_forward<DT, 7, false, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a); break;
        default:
            if (vec) hipExtLaunchKernelGGL((k_forward<DT, 8, true, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a);
            else hipExtLaunchKernelGGL((k_forward<DT, 8, false, MAXR, NC>), grid, block, 0, s, e0, e1, 0, a);
            break;
    }
}

template <bool MAXR, int NC>
void launch_dtype(const FwdArgs &a, int dtype, dim3 grid, int nch, bool vec, hipStream_t s,
                  hipEvent_t e0, hipEvent_t e1) {
    switch (dtype) {
        case BEVPOOL_F32: launch_nch<BEVPOOL_F32, MAXR, NC>(a, grid, nch, vec, s, e0, e1); break;
        case BEVPOOL_BF16: launch_nch<BEVPOOL_BF16, MAXR, NC>(a, grid, nch, vec, s, e0, e1); break;
        default: launch_nch<BEVPOOL_F16, MAXR, NC>(a, grid, nch, vec, s, e0, e1); break;
    }
}

}  // namespace
}  // namespace bevpool

using namespace bevpool;

int bevpool_launch_forward(const void *P, const void *F, const bevpool_plan_s *plan, float *out,
                           int64_t ldo, int32_t batch, int32_t channels, int32_t dtype,
                           int32_t reduce, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
    const bevpool_geometry &g = plan->geom;
    const int64_t n_pix = int64_t(g.n_cams) * g.feat_h * g.feat_w;
    const int64_t esize = dtype == BEVPOOL_F32 ? 4 : 2;
    const int64_t p_bytes = plan->n_points * esize;
    const int64_t f_bytes = n_pix * channels * esize;
    const int64_t o_bytes = int64_t(plan->n_cells) * ldo * 4;
    const int64_t run_bytes = int64_t(plan->n_runs) * 16;
    constexpr int64_t kLimit = int64_t(1) << 31;
    if (p_bytes >= kLimit || f_bytes >= kLimit || o_bytes >= kLimit || run_bytes >= kLimit)
        return bevpool_fail(BEVPOOL_ERR_OVERFLOW,
                            "channels=%d, row stride %lld: one frame's depth (%lld B), feature "
                            "(%lld B) or BEV (%lld B) tensor reaches 2 GiB", channels,
                            (long long)ldo, (long long)p_bytes, (long long)f_bytes,
                            (long long)o_bytes);
    if (batch > 65535)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "batch=%d exceeds 65535 frames per call", batch);

    // Generic cells: equal channel slices of at most kSliceChannels; slices
    // of 128, 80 or 64 when they divide C, whose rows move as 16-byte lanes.
    int slice_c;
    if (channels % 128 == 0) slice_c = 128;
    else if (channels % 80 == 0) slice_c = 80;
    else if (channels % 64 == 0) slice_c = 64;
    else slice_c = (channels + (channels + kSliceChannels - 1) / kSliceChannels - 1) /
                   ((channels + kSliceChannels - 1) / kSliceChannels);
    const int n_slices = (channels + slice_c - 1) / slice_c;
    const int nch = (slice_c + 15) / 16;

    FwdArgs a;
    a.P = static_cast<const char *>(P);
    a.F = static_cast<const char *>(F);
    a.out = out;
    a.table = plan->column_table;
    a.gen_hdr = plan->generic_hdr;
    a.gen_runs = plan->generic_runs;
    a.empty_cells = plan->empty_cells;
    a.cell_start = plan->cell_start;
    a.N = g.n_cams;
    a.D = g.n_depth;
    a.H = g.feat_h;
    a.W = g.feat_w;
    a.HW = g.feat_h * g.feat_w;
    a.C = channels;
    a.n_cells = plan->n_cells;
    a.ldo = int32_t(ldo);
    a.mean = reduce == BEVPOOL_MEAN ? 1 : 0;
    a.p_bytes = uint32_t(p_bytes);
    a.f_bytes = uint32_t(f_bytes);
    a.o_bytes = uint32_t(o_bytes);
    a.run_bytes = uint32_t(run_bytes);
    a.table_bytes = uint32_t(int64_t(g.n_cams) * g.n_depth * g.feat_w * 8);
    a.empty_bytes = uint32_t(int64_t(plan->n_empty) * 4);
    const bool out_aligned = ldo % 4 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0;
    a.vec_out = out_aligned ? 1 : 0;

    // sweep workgroups: only when some cell is swept
    a.n_dt = (g.n_depth + kSweepDepths - 1) / kSweepDepths;
    a.n_ct = (channels + kSweepChannels - 1) / kSweepChannels;
    a.rows = bevpool_sweep_rows(g.feat_w, g.feat_h);
    a.n_sweep = (plan->sweep_ok && plan->n_column > 0 && a.rows > 0) ? g.n_cams * a.n_dt * a.n_ct : 0;
    if (a.rows <= 0) a.rows = 4;
    a.n_chunks = (g.feat_h + a.rows - 1) / a.rows;
    a.ds = (a.rows * g.feat_w) | 1;   // odd depth-bin stride of the staged probabilities
    a.waves = g.feat_w < kSweepWaves ? g.feat_w : kSweepWaves;

    a.n_heavy = plan->n_generic_heavy;
    a.n_light = plan->n_run_cells - plan->n_generic_heavy;
    a.cc_hdr = plan->cc_hdr;
    a.cc_list = plan->cc_list;
    a.n_cc = plan->n_combo_cells;
    a.cc_bytes = uint32_t(int64_t(plan->n_cc_combos) * 8);
    a.div_w = make_fastdiv(uint32_t(g.feat_w));
    a.div_d = make_fastdiv(uint32_t(g.n_depth));
    a.slice_c = slice_c;
    a.n_slices = n_slices;
    a.n_empty = plan->n_empty;
    a.zero_vec = (channels % 4 == 0 && out_aligned) ? 1 : 0;
    a.zero_units = a.zero_vec ? channels / 4 : channels;
    a.row_units = a.zero_vec ? int32_t(ldo / 4) : int32_t(ldo);
    a.div_units = make_fastdiv(uint32_t(a.zero_units));

    int G = plan->n_cus > 0 ? plan->n_cus : 256;
    if (a.n_sweep > G) G = a.n_sweep;
    const dim3 grid(G, batch);
    // 4-element lanes for generic cells: every row slice of F (elements) and
    // of the output (fp32) starts on a 4-element boundary of an aligned
    // buffer (slices of 65..80 channels, or exactly 64 or 128)
    const bool aligned = out_aligned && reinterpret_cast<uintptr_t>(F) % (4 * esize) == 0;
    const bool vec = aligned && ((nch == 5 && channels % 4 == 0 && slice_c % 4 == 0) ||
                                 (nch == 4 && slice_c == 64 && channels % 64 == 0) ||
                                 (nch == 8 && slice_c == 128 && channels % 128 == 0));
    const bool maxr = reduce == BEVPOOL_MAX;
    // 8 staged rows go with at most 6 columns a wave (two steps of 4 rows);
    // otherwise 4 rows and up to kSweepMaxCols columns
    const bool wide = a.rows != 8;
    if (maxr && wide) launch_dtype<true, kSweepMaxCols>(a, dtype, grid, nch, vec, stream, start, stop);
    else if (maxr) launch_dtype<true, 6>(a, dtype, grid, nch, vec, stream, start, stop);
    else if (wide) launch_dtype<false, kSweepMaxCols>(a, dtype, grid, nch, vec, stream, start, stop);
    else launch_dtype<false, 6>(a, dtype, grid, nch, vec, stream, start, stop);
    BEVPOOL_HIP(hipGetLastError());
    return BEVPOOL_OK;
}
