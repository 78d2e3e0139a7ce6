// Per-frame BEV pooling: fused lift (depth probability x feature) and
// per-cell sum (BEVFusion, arXiv 2205.13542, Sec. III-B, first paragraph and
// "Interval Reduction"). The paper gives each cell one GPU thread that walks
// the cell's interval. Here the work follows the camera geometry instead
// (see the partition in internal.h): a launch with four workgroup roles,
// and a second one when the plan has multi-combo cells.
//
//   column items   kColDepth depth bins x kColWidth pixel columns of one
//                  camera. A group of 16 lanes (one DPP row) owns a column
//                  and holds kColDepth fp32 accumulators per channel. Each
//                  feature row (n, h, w) is read once and applied to every
//                  depth bin of the item; the depth probabilities are read
//                  one per lane and broadcast to the group through LDS.
//                  Single-combo cells are stored from registers; each
//                  combo of a multi-combo cell stores its sum in the
//                  borrowed row of its partial slot.
//   light generic  one wave per generic cell. Its runs (consecutive depth
//                  bins of one pixel) are taken 64 at a time: each lane loads
//                  one run record and sums the run's depth probabilities,
//                  then the four lane groups share the runs out, each run
//                  costing one feature row. Groups are combined by shuffles.
//   heavy generic  one workgroup per generic cell with more than kGenHeavy
//                  points; its waves take the 64-run chunks in turn, and the
//                  workgroup's lane groups are combined through LDS.
//   zero rows      cells without points, one per thread of a workgroup,
//                  as one flat run of 16-byte stores over their rows (only
//                  when there is no second launch).
//
// The second launch, k_combine, adds each multi-combo cell's partial slots
// in slot order, zeroes the borrowed rows, and zeroes the other empty rows.
// The zeroing is bandwidth-bound work that covers the latency of the slot
// reads, and the first launch, whose column items are latency-bound, runs
// without write traffic beside it. The column items also read the plan
// arrays that the second launch starts from (the empty-cell list and the
// multi-combo records) once, so that those first loads of the second launch
// are served from the caches rather than from HBM.
//
// Channels go across the 16 lanes of a group (channel j + 16k in lane j, or
// 16-byte lanes for aligned slices of 64, 65..80 or 128 channels), so every
// load and store of a row is contiguous across the group. Rows wider than
// kSliceChannels are done in slices (grid z).
//
// All reads and writes of P, F and the BEV map go through buffer resources
// of one frame each. An access that must not happen gets an offset past the
// end of its buffer: the hardware range check then returns 0 for a load and
// drops a store, so the hot loops carry no branches for bounds or masks.
//
// The same kernels take the mean and the max (the "Interval Reduction"
// paragraph names both besides the sum). Mean: sums as above, each final
// value divided by its cell's point count where it is stored (a single
// combo's count is its row range; other cells read the interval table).
// Max (template flag MAXR): the FMAs become max(acc, p * f) from -inf, a
// masked row carries a NaN probability that fmaxf ignores, and partial slots
// are combined by max. Rows of the map are ldo floats apart (ldo >= C), so a
// call can fill one channel block of a wider map, e.g. one z slab.
//
// Each output row gets its final value from one plain store (a borrowed row
// holds a partial sum before it is zeroed), and every sum runs in an order
// fixed by the plan, so results are deterministic. The per-row products are
// small (kColDepth bins x a row slice) and done with FMAs: the column items
// are bound by memory latency, not by arithmetic.
#include <math.h>
#include <stdint.h>

#include <hip/hip_ext.h>

#include <type_traits>

#include "device.h"
#include "internal.h"

namespace bevpool {
namespace {


// Rows of empty cells to zero: entries zero_begin .. zero_end-1 of the
// empty-cell list.
struct ZeroArgs {
    float *out;
    const int32_t *empty_cells;
    int32_t n_cells, ldo;               // output rows are ldo floats apart
    int32_t zero_begin, zero_end;
    int32_t zero_vec, zero_units;       // float4 units (or floats) per row
    int32_t row_units;                  // the same units from one row to the next
    FastDiv div_units;
};

struct FwdArgs {
    const char *P, *F;
    float *out;
    const int2 *table;
    const int4 *gen_hdr;
    const int4 *gen_runs;
    int32_t N, D, H, W, HW;
    int32_t n_cells, C, slice_c;
    int32_t ldo, mean;                  // output row stride (floats); divide sums by counts
    const int32_t *cell_start;          // interval table: point counts of the cells
    uint32_t p_bytes, f_bytes, o_bytes, run_bytes;   // per frame (runs: whole table)
    int32_t items_d, items_w, n_items;
    int32_t n_planes, plane;            // column-table planes in use, entries per plane
    int32_t n_heavy, n_light;
    int32_t base_col, base_zero, base_light;
    ZeroArgs zero;
    // plan arrays read first by the second launch; the column items of
    // frame 0, slice 0 touch them (kWarmArrays arrays of warm_n[i] words)
    const int32_t *warm[4];
    int32_t warm_n[4];
};
constexpr int kWarmArrays = 4;

// The buffers of frame b: depth probabilities, features, BEV map.
struct Frame {
    Rsrc P, F, O;
    __device__ __forceinline__ Frame(const FwdArgs &a, int b)
        : P(make_rsrc(a.P + int64_t(b) * a.p_bytes, a.p_bytes)),
          F(make_rsrc(a.F + int64_t(b) * a.f_bytes, a.f_bytes)),
          O(make_rsrc(reinterpret_cast<const char *>(a.out) + int64_t(b) * a.o_bytes, a.o_bytes)) {}
};

constexpr int kStages = 4;                      // row-pair stages in flight per wave

// LDS row stride of a lane group's partial sums: 16*NCH floats, padded so
// that the four groups of a wave start on different bank quarters.
template <int NCH>
constexpr int slot_stride() { return 16 * NCH + ((NCH % 2 == 0) ? 16 : 0); }


// Column items in (camera, column block, depth block) order are placed so
// that consecutive depth blocks of one column block share an XCD's L2 and,
// three at a time, a CU's L1 (xcd_cu_remap in device.h).
constexpr int kCuRounds = 3;


// Two feature rows of a column and the lane's depth probability for them.
template <int NCH>
struct Stage {
    float pv;
    Row<NCH> f0, f1;
};


// acc[J] += pb[J] * f for the kColDepth depth bins of one row: pb holds the
// row's probabilities of this lane group's column, read back from LDS as
// broadcasts (a DPP broadcast operand would halve the FMA issue rate).
// With MAXR, acc[J] = max(acc[J], pb[J] * f) instead: a masked-off row
// carries a NaN probability, and fmaxf ignores the NaN product.
template <int NCH, bool MAXR>
__device__ __forceinline__ void apply_row(float (&acc)[kColDepth][NCH], const float4 &lo,
                                          const float4 &hi, const Row<NCH> &f) {
    const float pb[kColDepth] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
    for (int J = 0; J < kColDepth; ++J)
#pragma unroll
        for (int k = 0; k < NCH; ++k) {
            if constexpr (MAXR)
                acc[J][k] = fmaxf(acc[J][k], pb[J] * f.v[k]);
            else
                acc[J][k] = __builtin_fmaf(pb[J], f.v[k], acc[J][k]);
        }
}

// After the row loop: each depth bin's sums go to the BEV row named by its
// table entry: its single-combo cell, or the borrowed empty-cell row that
// holds the partial sum of its combo. Lane J of the group holds the entry of
// depth bin J. For the mean, a single-combo cell's sum is divided by its
// point count, the combo's row range; partial sums are divided later.
template <int J, int NCH, bool VEC>
struct Emit {
    static __device__ __forceinline__ void run(const float (&acc)[kColDepth][NCH], int ex, int ey,
                                               uint32_t dm, Rsrc out, uint32_t ch_off, int ldo,
                                               bool mean, bool tail_ok) {
        if (dm & (1u << J)) {
            const int x = row_bcast<J>(ex);
            float v[NCH];
#pragma unroll
            for (int k = 0; k < NCH; ++k) v[k] = acc[J][k];
            if (mean) {
                const uint32_t y = uint32_t(row_bcast<J>(ey));
                if (!(y & kComboMulti)) {
                    const float cnt = float(int((y >> 16) & 0x3FFFu) - int(y & 0xFFFFu));
#pragma unroll
                    for (int k = 0; k < NCH; ++k) v[k] = v[k] / cnt;
                }
            }
            store_row<NCH, VEC>(out, x >= 0 ? uint32_t(x) * uint32_t(ldo) * 4u + ch_off : kOff, v,
                           tail_ok);
        }
        Emit<J + 1, NCH, VEC>::run(acc, ex, ey, dm, out, ch_off, ldo, mean, tail_ok);
    }
};
template <int NCH, bool VEC>
struct Emit<kColDepth, NCH, VEC> {
    static __device__ __forceinline__ void run(const float (&)[kColDepth][NCH], int, int, uint32_t,
                                               Rsrc, uint32_t, int, bool, bool) {}
};

// Zeroing workgroup zb of BS threads: the rows of BS listed empty cells of
// frame b, from entry z.zero_begin + zb * BS on, written as one flat
// sequence of 16-byte (or 4-byte) units: unit f is unit f % U of row f / U
// (a row's first U units; rows are row_units apart).
// Rows of consecutive cells are adjacent in memory, so runs of empty cells
// become contiguous stores. The cell ids are staged in LDS first, so no
// store waits on a load.
template <int BS>
__device__ void zero_rows(const ZeroArgs &z, int zb, int b, int *s_cell) {
    const int e0 = z.zero_begin + zb * BS;
    const int ne = min(BS, z.zero_end - e0);
    if (int(threadIdx.x) < ne) s_cell[threadIdx.x] = z.empty_cells[e0 + threadIdx.x];
    __syncthreads();
    const int U = z.zero_units;
    const int total = ne * U;
    const int RU = z.row_units;
    if (z.zero_vec) {
        float4 *o = reinterpret_cast<float4 *>(z.out + int64_t(b) * z.n_cells * z.ldo);
        for (int f = threadIdx.x; f < total; f += BS) {
            const int r = int(fdiv(uint32_t(f), z.div_units));
            o[int64_t(s_cell[r]) * RU + (f - r * U)] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
    } else {
        float *o = z.out + int64_t(b) * z.n_cells * z.ldo;
        for (int f = threadIdx.x; f < total; f += BS) {
            const int r = int(fdiv(uint32_t(f), z.div_units));
            o[int64_t(s_cell[r]) * RU + (f - r * U)] = 0.f;
        }
    }
}

// fn(integral_constant<int, I>) for I = B .. E-1, each I a constant
// expression (for the DPP lane selects).
template <int B, int E, typename Fn>
__device__ __forceinline__ void static_for(Fn &&fn) {
    if constexpr (B < E) {
        fn(std::integral_constant<int, B>());
        static_for<B + 1, E>(fn);
    }
}

// Zeroing workgroups of BS threads needed for the entries of z.
template <int BS>
int zero_blocks(const ZeroArgs &z) { return (z.zero_end - z.zero_begin + BS - 1) / BS; }

template <int DT, int NCH, bool VEC, bool MAXR, bool SEG>
__device__ void column_item(const FwdArgs &a, const Frame &fr, int item, int c0, int cn,
                            float *s_pb) {
    constexpr uint32_t ES = Elem<DT>::kBytes;
    const int db = item % a.items_d;
    const int t = item / a.items_d;
    const int wb = t % a.items_w, n = t / a.items_w;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15;
    const int wl = wave * 4 + (lane >> 4);        // column within the item
    const int w = wb * kColWidth + wl;
    const int jd = j & 7;
    const int d = db * kColDepth + jd;
    const bool in_w = w < a.W;
    const bool tail_ok = j + 16 * (NCH - 1) < cn;

    // The row loop covers all H rows, so its loads need nothing from the
    // column table and the first stages are issued before the entries
    // arrive; a lane's probability is masked to its combo's row range when
    // its stage is applied.
    const bool dw_ok = in_w && d < a.D;
    const uint32_t p_col = dw_ok ? uint32_t(((n * a.D + d) * a.H) * a.W + w) * ES : kOff;
    const uint32_t p_row = uint32_t(a.W) * ES;
    const uint32_t f_col = in_w ? (uint32_t(n * a.HW + w) * uint32_t(a.C) + uint32_t(c0)) * ES : kOff;
    const uint32_t f_row = uint32_t(a.W) * uint32_t(a.C) * ES;
    const int hsel = j >> 3;
    const int H = a.H;
    auto load_stage = [&](Stage<NCH> &st, int h) {
        st.pv = Elem<DT>::load(fr.P, h + hsel < H ? p_col + uint32_t(h + hsel) * p_row : kOff);
        load_row<DT, NCH, VEC>(st.f0, fr.F, h < H ? f_col + uint32_t(h) * f_row : kOff);
        load_row<DT, NCH, VEC>(st.f1, fr.F, h + 1 < H ? f_col + uint32_t(h + 1) * f_row : kOff);
    };
    // plane 0 of the column table holds each combo's first row segment (the
    // whole combo on a level rig); plane s its segment s, done in pass s
    const int64_t tab0 = (int64_t(n) * a.D + d) * a.W + w;
    int2 e = make_int2(-1, 0);
    if (dw_ok) e = a.table[tab0];
    Stage<NCH> st[kStages];
    // Issued stage by stage, in the order in which the loop consumes them:
    // the loop's waits count outstanding loads in issue order, and a
    // prologue reordered by the scheduler would make every iteration wait
    // for nearly all of them.
#pragma unroll
    for (int u = 0; u < kStages; ++u) {
        load_stage(st[u], 2 * u);
        __builtin_amdgcn_sched_barrier(0);
    }

    // Touch the second launch's plan arrays (after this item's own loads):
    // item i reads words i * kFwdBlock + t, i * kFwdBlock + t + kFwdBlock *
    // n_items, ... of each. The values are only kept live until the end.
    // The first word of each array is loaded without a wait (an offset past
    // the array reads 0) and consumed only at the end; further words (grids
    // with more plan entries than threads) are read in a loop.
    int warm = 0;
    int wfirst[kWarmArrays];
#pragma unroll
    for (int q = 0; q < kWarmArrays; ++q) wfirst[q] = 0;
    if (blockIdx.y == 0 && blockIdx.z == 0) {
        const int stride = a.n_items * kFwdBlock;
        const int i0 = item * kFwdBlock + int(threadIdx.x);
#pragma unroll
        for (int q = 0; q < kWarmArrays; ++q) {
            const Rsrc wr = make_rsrc(a.warm[q], uint32_t(a.warm_n[q]) * 4u);
            wfirst[q] = int(__builtin_amdgcn_raw_buffer_load_b32(wr, i0 < a.warm_n[q] ? i0 * 4 : int(kOff), 0, 0));
        }
#pragma unroll
        for (int q = 0; q < kWarmArrays; ++q)
            for (int i = i0 + stride; i < a.warm_n[q]; i += stride) warm ^= a.warm[q][i];
    }

    // Row segments (SEG): a combo whose kept rows fall into several cells
    // has one segment per cell, ascending and disjoint, segment s in plane s
    // of the table. One sweep over the rows serves them all: a lane masks
    // its probability to the segment that holds its row, and when the rows
    // pass the end of a segment that is not its combo's last, the depth
    // bin's sums go to that segment's row and start again from zero. The
    // last segment is emitted after the loop like a whole combo.
    // A segment whose cell is gathered (demoted to a generic cell) has no
    // entry: the list is compacted to the served segments, whose rows the
    // sweep masks and flushes; rows of the others stay masked.
    int2 seg[SEG ? kMaxSeg : 1];
    int nseg = e.x >= 0 ? 1 : 0;
    seg[0] = e;
    if constexpr (SEG) {
#pragma unroll
        for (int q = 1; q < kMaxSeg; ++q) seg[q] = make_int2(-1, 0);
#pragma unroll
        for (int q = 1; q < kMaxSeg; ++q) {
            const int2 eq = (dw_ok && q < a.n_planes) ? a.table[int64_t(q) * a.plane + tab0]
                                                      : make_int2(-1, 0);
            if (eq.x >= 0) {
#pragma unroll
                for (int i = 0; i < kMaxSeg; ++i) seg[i] = i == nseg ? eq : seg[i];
                ++nseg;
            }
        }
    }
    // the lane's current segment for masking, and the next segment to flush
    int cur = 0, fl = 0;
    auto seg_lo = [&](int q) {
        int v = 0;
#pragma unroll
        for (int i = 0; i < (SEG ? kMaxSeg : 1); ++i) v = i == q ? int(uint32_t(seg[i].y) & 0xFFFFu) : v;
        return v;
    };
    auto seg_hi = [&](int q) {
        int v = 0;
#pragma unroll
        for (int i = 0; i < (SEG ? kMaxSeg : 1); ++i) v = i == q ? int((uint32_t(seg[i].y) >> 16) & 0x3FFFu) : v;
        return v;
    };
    auto seg_entry = [&](int q) {
        int2 v = make_int2(-1, 0);
#pragma unroll
        for (int i = 0; i < (SEG ? kMaxSeg : 1); ++i) v = i == q ? seg[i] : v;
        return v;
    };
    // row after which segment fl ends, if it is not the last one
    auto flush_row = [&]() { return fl + 1 < nseg ? seg_hi(fl) - 1 : 0x7FFFFFFF; };
    const bool act = nseg > 0;
    // the whole combo's rows (one plane)
    const uint32_t ey0 = uint32_t(e.y);
    const int hlo = act ? int(ey0 & 0xFFFFu) : 0x7FFFFFFF;
    const int hhi = act ? int((ey0 >> 16) & 0x3FFFu) : 0;
    // depth bins present in the wave (a wave without any skips the loop)
    const uint64_t bal = __ballot(act);
    const uint32_t dm = uint32_t((bal | (bal >> 16) | (bal >> 32) | (bal >> 48)) & 0xFFu);

    float acc[kColDepth][NCH];
#pragma unroll
    for (int q = 0; q < kColDepth; ++q)
#pragma unroll
        for (int k = 0; k < NCH; ++k) acc[q][k] = MAXR ? -INFINITY : 0.f;
    const float masked = MAXR ? __builtin_nanf("") : 0.f;   // probability of a row outside the combo
    const bool mean = !MAXR && a.mean != 0;

    // depth bin J's sums to the row of its segment that ends at row r, if
    // one does (lane J of the group knows), then from zero again
    auto flush = [&](int r) {
        const int my = flush_row();
        static_for<0, kColDepth>([&](auto Jc) {
            constexpr int J = decltype(Jc)::value;
            if (row_bcast<J>(my) == r) {
                const int2 fe = seg_entry(fl);
                const int x = row_bcast<J>(fe.x);
                const uint32_t y = uint32_t(row_bcast<J>(fe.y));
                float v[NCH];
#pragma unroll
                for (int k = 0; k < NCH; ++k) v[k] = acc[J][k];
                if (mean && !(y & kComboMulti)) {
                    const float cnt = float(int((y >> 16) & 0x3FFFu) - int(y & 0xFFFFu));
#pragma unroll
                    for (int k = 0; k < NCH; ++k) v[k] = v[k] / cnt;
                }
                store_row<NCH, VEC>(fr.O, x >= 0 ? uint32_t(x) * uint32_t(a.ldo) * 4u + uint32_t(c0) * 4u : kOff,
                                    v, tail_ok);
#pragma unroll
                for (int k = 0; k < NCH; ++k) acc[J][k] = MAXR ? -INFINITY : 0.f;
            }
        });
        if (my == r) ++fl;
    };

    if (dm != 0) {
        // A ring of kStages stages of two rows: while one stage is applied,
        // the loads of the next kStages - 1 are outstanding. Each lane's
        // masked probability (depth bin j & 7, row j >> 3 of the stage) goes
        // through this group's 16 LDS words and comes back to all 16 lanes.
        // Every pass runs all kStages stages: rows past H load nothing and
        // add zeros, so the loop has one exit and its waits hold in steady
        // state.
        float *pq = s_pb + (wave * 4 + (lane >> 4)) * 16;
        for (int h = 0; h < H; h += 2 * kStages) {
#pragma unroll
            for (int u = 0; u < kStages; ++u) {
                const int hs = h + 2 * u;
                const int hp = hs + hsel;
                bool keep;
                if constexpr (SEG) {
                    while (cur + 1 < nseg && hp >= seg_hi(cur)) ++cur;
                    keep = hp >= seg_lo(cur) && hp < seg_hi(cur);
                } else {
                    keep = hp >= hlo && hp < hhi;
                }
                pq[j] = keep ? st[u].pv : masked;
                __builtin_amdgcn_wave_barrier();
                const float4 r0a = *reinterpret_cast<const float4 *>(pq);
                const float4 r0b = *reinterpret_cast<const float4 *>(pq + 4);
                const float4 r1a = *reinterpret_cast<const float4 *>(pq + 8);
                const float4 r1b = *reinterpret_cast<const float4 *>(pq + 12);
                __builtin_amdgcn_wave_barrier();
                // a segment of some lane's combo ends in this stage
                const bool split = SEG && __ballot(flush_row() <= hs + 1) != 0;
                apply_row<NCH, MAXR>(acc, r0a, r0b, st[u].f0);
                if (split) flush(hs);
                apply_row<NCH, MAXR>(acc, r1a, r1b, st[u].f1);
                if (split) flush(hs + 1);
                load_stage(st[u], hs + 2 * kStages);
            }
        }
    }

    // the combo's last segment (the whole combo when it has one)
    if constexpr (SEG) {
        const int2 el = seg_entry(nseg > 0 ? nseg - 1 : 0);
        Emit<0, NCH, VEC>::run(acc, el.x, el.y, dm, fr.O, uint32_t(c0) * 4u, a.ldo, mean, tail_ok);
    } else {
        Emit<0, NCH, VEC>::run(acc, e.x, e.y, dm, fr.O, uint32_t(c0) * 4u, a.ldo, mean, tail_ok);
    }
    asm volatile("" ::"v"(warm ^ wfirst[0] ^ wfirst[1] ^ wfirst[2] ^ wfirst[3]));   // only loaded, not needed
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
        for (int q = 0; q < len; ++q) {
            const float pq = Elem<DT>::load(fr.P, uint32_t(p0 + q * a.HW) * ES);
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
    generic_runs<DT, NCH, VEC, MAXR>(acc, a, fr, hdr, c0, wave, kFwdWaves);
#pragma unroll
    for (int q = 0; q < NCH; ++q) s_part[wl * SS + j + 16 * q] = acc[q];
    __syncthreads();
    if (wl == 0) {
        float sum[NCH];
#pragma unroll
        for (int q = 0; q < NCH; ++q) sum[q] = MAXR ? -INFINITY : 0.f;
        for (int g = 0; g < kColWidth; ++g)
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
}

template <int DT, int NCH, bool VEC, bool MAXR, bool SEG>
__global__ __launch_bounds__(kFwdBlock) void k_forward(FwdArgs a) {
    __shared__ float s_part[kColWidth * slot_stride<NCH>()];   // heavy cells: group partials
    __shared__ int s_cell[kFwdBlock];                          // zero rows: cell ids
    __shared__ __align__(16) float s_pb[kFwdBlock];   // probability broadcast: 16 words per lane group
    const int bx = blockIdx.x, b = blockIdx.y;
    const int c0 = blockIdx.z * a.slice_c;
    const int cn = min(a.slice_c, a.C - c0);
    if (bx < a.n_heavy) {
        heavy_generic<DT, NCH, VEC, MAXR>(a, Frame(a, b), bx, c0, cn, s_part);
    } else if (bx < a.base_col) {
        return;  // padding: column items start on a multiple of 8
    } else if (bx < a.base_col + a.n_items) {
        column_item<DT, NCH, VEC, MAXR, SEG>(a, Frame(a, b), xcd_cu_remap<kCuRounds>(bx - a.base_col, a.n_items),
                                        c0, cn, s_pb);
    } else if (bx < a.base_zero) {
        return;
    } else if (bx < a.base_light) {
        if (blockIdx.z == 0) zero_rows<kFwdBlock>(a.zero, bx - a.base_zero, b, s_cell);   // whole rows
    } else {
        const int k = (bx - a.base_light) * kFwdWaves + int(threadIdx.x >> 6);
        if (k < a.n_light) light_generic<DT, NCH, VEC, MAXR>(a, Frame(a, b), k, c0, cn);
    }
}

// Cells fed by several combos: the slots of multi-combo cell k are
// multi_begin[k] .. multi_begin[k+1]-1, slot s held in the BEV row of empty
// cell empty_cells[s]; the rows of the first kCombineInline slots are also
// listed in multi_rows[k], so one round of loads finds the cell, its slot
// count and those rows. The slots are added in slot order into the cell's
// row, and the borrowed rows are zeroed. One group of 16 lanes per cell,
// channels j, j + 16, ... The last n_zblocks workgroups zero empty rows
// instead: the combine workgroups are dispatched first, so their two rounds
// of loads (records, then slot rows; both cached, see the column items) are
// issued before the bandwidth-bound zero stores, which then cover them.
constexpr int kCombineChunks = 5;   // 16-channel chunks per pass (80 channels)
constexpr int kCombineGroups = kBlock / 16;   // cells per workgroup
static_assert(kCombineInline <= 16, "inline rows come from one lane each of a 16-lane group");

struct CombineArgs {
    float *out;
    const int32_t *multi_begin, *multi_cell, *multi_rows, *empty_cells;
    const int32_t *cell_start;
    int32_t n_multi, C, ldo, mean, n_zblocks;
    uint32_t o_bytes;
    ZeroArgs zero;
};

// Row of slot sl + U of this lane group's cell (held by its lane U), as a
// byte offset, or kOff past the cell's last slot.
template <int U>
__device__ __forceinline__ uint32_t slot_row(int r, int sl, int n, uint32_t row_bytes) {
    const int x = row_bcast<U>(r);
    return sl + U < n ? uint32_t(x) * row_bytes : kOff;
}

template <int U>
struct SlotRows {
    static __device__ __forceinline__ void run(uint32_t *rb, int r, int sl, int n, uint32_t row_bytes) {
        rb[U] = slot_row<U>(r, sl, n, row_bytes);
        SlotRows<U + 1>::run(rb, r, sl, n, row_bytes);
    }
};
template <>
struct SlotRows<kCombineInline> {
    static __device__ __forceinline__ void run(uint32_t *, int, int, int, uint32_t) {}
};

// With MAXR the slots' largest value is taken instead of their sum; for the
// mean the sum is divided by the cell's point count. With VEC (every
// 80-channel pass of the row holds 65..80 channels, rows on 16-byte
// boundaries) a lane moves channels 4j..4j+3 as one 16-byte access and
// channel 64 + j as one 4-byte access; otherwise channels j + 16k.
template <bool MAXR, bool VEC>
__global__ __launch_bounds__(kBlock) void k_combine(CombineArgs a) {
    __shared__ int s_cell[kBlock];
    const int b = blockIdx.y;
    const int n_cblocks = int(gridDim.x) - a.n_zblocks;
    if (int(blockIdx.x) >= n_cblocks) {
        zero_rows<kBlock>(a.zero, int(blockIdx.x) - n_cblocks, b, s_cell);
        return;
    }
    const int k = int(blockIdx.x) * kCombineGroups + int(threadIdx.x >> 4);
    if (k >= a.n_multi) return;
    const int j = threadIdx.x & 15;
    const int ji = j % kCombineInline;
    const Rsrc O = make_rsrc(reinterpret_cast<const char *>(a.out) + int64_t(b) * a.o_bytes, a.o_bytes);
    // one round: inline rows (lane u holds slot u), the cell, the slot range
    const int r_inline = a.multi_rows[int64_t(k) * kCombineInline + ji];
    const int s0 = a.multi_begin[k];
    const int n = a.multi_begin[k + 1] - s0;
    const uint32_t row = uint32_t(a.ldo) * 4u;
    const int cell = a.multi_cell[k];
    const uint32_t obase = uint32_t(cell) * row;
    const float cnt = (!MAXR && a.mean) ? float(a.cell_start[cell + 1] - a.cell_start[cell]) : 1.f;
    // every lane of the group runs every pass (the slot rows are exchanged
    // between its lanes); channels past C are masked
    for (int cb = 0; cb < a.C; cb += kCombineChunks * 16) {
        const int cn = min(kCombineChunks * 16, a.C - cb);
        const uint32_t cboff = uint32_t(cb) * 4u;
        Row<kCombineChunks> sum;
#pragma unroll
        for (int q = 0; q < kCombineChunks; ++q) sum.v[q] = MAXR ? -INFINITY : 0.f;
        // kCombineInline slots' loads in flight at a time, added in slot order
        for (int sl = 0; sl < n; sl += kCombineInline) {
            const int r = sl == 0 ? r_inline : (sl + ji < n ? a.empty_cells[s0 + sl + ji] : 0);
            uint32_t rb[kCombineInline];
            SlotRows<0>::run(rb, r, sl, n, row);
            Row<kCombineChunks> v[kCombineInline];
#pragma unroll
            for (int u = 0; u < kCombineInline; ++u) {
                if constexpr (VEC) {
                    load_row<BEVPOOL_F32, kCombineChunks, true>(v[u], O, rb[u] + cboff);
                } else {
#pragma unroll
                    for (int q = 0; q < kCombineChunks; ++q)
                        v[u].v[q] = Elem<BEVPOOL_F32>::load(
                            O, j + 16 * q < cn ? rb[u] + cboff + uint32_t(j + 16 * q) * 4u : kOff);
                }
            }
#pragma unroll
            for (int u = 0; u < kCombineInline; ++u)
#pragma unroll
                for (int q = 0; q < kCombineChunks; ++q)
                    if (sl + u < n) sum.v[q] = MAXR ? fmaxf(sum.v[q], v[u].v[q]) : sum.v[q] + v[u].v[q];
            const float zero[kCombineChunks] = {0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int u = 0; u < kCombineInline; ++u) {
                if constexpr (VEC) {
                    store_row<kCombineChunks, true>(O, rb[u] + cboff, zero, 64 + j < cn);
                } else {
#pragma unroll
                    for (int q = 0; q < kCombineChunks; ++q)
                        store_f32(O, j + 16 * q < cn ? rb[u] + cboff + uint32_t(j + 16 * q) * 4u : kOff, 0.f);
                }
            }
        }
        if (!MAXR && a.mean) {
#pragma unroll
            for (int q = 0; q < kCombineChunks; ++q) sum.v[q] = sum.v[q] / cnt;
        }
        if constexpr (VEC) {
            store_row<kCombineChunks, true>(O, obase + cboff, sum.v, 64 + j < cn);
        } else {
#pragma unroll
            for (int q = 0; q < kCombineChunks; ++q)
                store_f32(O, j + 16 * q < cn ? obase + cboff + uint32_t(j + 16 * q) * 4u : kOff, sum.v[q]);
        }
    }
}

// Kernel-boundary events (either may be null): they take the timestamps of
// the dispatch itself rather than of separate queue entries.
template <int DT, bool MAXR, bool SEG>
void launch_dtype(const FwdArgs &a, dim3 grid, int nch, bool vec, hipStream_t s, hipEvent_t e0,
                  hipEvent_t e1) {
    const dim3 block(kFwdBlock);
    switch (nch) {
        case 1: hipExtLaunchKernelGGL((k_forward<DT, 1, false, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a); break;
        case 2: hipExtLaunchKernelGGL((k_forward<DT, 2, false, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a); break;
        case 3: hipExtLaunchKernelGGL((k_forward<DT, 3, false, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a); break;
        case 4:
            if (vec) hipExtLaunchKernelGGL((k_forward<DT, 4, true, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a);
            else hipExtLaunchKernelGGL((k_forward<DT, 4, false, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a);
            break;
        case 5:
            if (vec) hipExtLaunchKernelGGL((k_forward<DT, 5, true, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a);
            else hipExtLaunchKernelGGL((k_forward<DT, 5, false, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a);
            break;
        case 6: hipExtLaunchKernelGGL((k_forward<DT, 6, false, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a); break;
        case 7: hipExtLaunchKernelGGL((k_forward<DT, 7, false, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a); break;
        default:
            if (vec) hipExtLaunchKernelGGL((k_forward<DT, 8, true, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a);
            else hipExtLaunchKernelGGL((k_forward<DT, 8, false, MAXR, SEG>), grid, block, 0, s, e0, e1, 0, a);
            break;
    }
}

template <bool MAXR, bool SEG>
void launch_forward(const FwdArgs &a, int dtype, dim3 grid, int nch, bool vec, hipStream_t s,
                    hipEvent_t e0, hipEvent_t e1) {
    switch (dtype) {
        case BEVPOOL_F32: launch_dtype<BEVPOOL_F32, MAXR, SEG>(a, grid, nch, vec, s, e0, e1); break;
        case BEVPOOL_BF16: launch_dtype<BEVPOOL_BF16, MAXR, SEG>(a, grid, nch, vec, s, e0, e1); break;
        default: launch_dtype<BEVPOOL_F16, MAXR, SEG>(a, grid, nch, vec, s, e0, e1); break;
    }
}

int round8(int x) { return (x + 7) & ~7; }

// Eighths of the unborrowed empty rows that the combine kernel zeroes.
constexpr int kZeroLate = 8;

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

    // Equal slices of at most kSliceChannels channels; slices of 128, 80 or
    // 64 when they divide C, whose rows move as 16-byte lanes.
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
    a.N = g.n_cams;
    a.D = g.n_depth;
    a.H = g.feat_h;
    a.W = g.feat_w;
    a.HW = g.feat_h * g.feat_w;
    a.n_cells = plan->n_cells;
    a.C = channels;
    a.slice_c = slice_c;
    a.ldo = int32_t(ldo);
    a.mean = reduce == BEVPOOL_MEAN ? 1 : 0;
    a.cell_start = plan->cell_start;
    a.p_bytes = uint32_t(p_bytes);
    a.f_bytes = uint32_t(f_bytes);
    a.o_bytes = uint32_t(o_bytes);
    a.run_bytes = uint32_t(run_bytes);
    a.items_d = (g.n_depth + kColDepth - 1) / kColDepth;
    a.items_w = (g.feat_w + kColWidth - 1) / kColWidth;
    a.n_items = g.n_cams * a.items_d * a.items_w;
    a.n_planes = plan->n_planes;
    a.plane = g.n_cams * g.n_depth * g.feat_w;
    a.n_heavy = plan->n_generic_heavy;
    a.n_light = plan->n_generic - plan->n_generic_heavy;

    // Empty rows: the first n_partials entries of the list are borrowed by
    // partial slots (the combine kernel zeroes them); of the rest, the
    // combine kernel, when there is one, takes the last kZeroLate / 8.
    const bool combine = plan->n_multi > 0;
    a.warm[0] = plan->empty_cells;
    a.warm_n[0] = combine ? plan->n_empty : 0;
    a.warm[1] = plan->multi_rows;
    a.warm_n[1] = combine ? plan->n_multi * kCombineInline : 0;
    a.warm[2] = plan->multi_begin;
    a.warm_n[2] = combine ? plan->n_multi + 1 : 0;
    a.warm[3] = plan->multi_cell;
    a.warm_n[3] = combine ? plan->n_multi : 0;
    ZeroArgs z;
    z.out = out;
    z.empty_cells = plan->empty_cells;
    z.n_cells = plan->n_cells;
    z.ldo = int32_t(ldo);
    z.zero_vec = (channels % 4 == 0 && ldo % 4 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0) ? 1 : 0;
    z.zero_units = z.zero_vec ? channels / 4 : channels;
    z.row_units = z.zero_vec ? int32_t(ldo / 4) : int32_t(ldo);
    z.div_units = make_fastdiv(uint32_t(z.zero_units));
    const int n_free = plan->n_empty - plan->n_partials;
    const int n_late = combine ? int(int64_t(n_free) * kZeroLate / 8) : 0;
    a.zero = z;
    a.zero.zero_begin = plan->n_partials;
    a.zero.zero_end = plan->n_empty - n_late;
    a.base_col = round8(a.n_heavy);
    a.base_zero = round8(a.base_col + a.n_items);
    a.base_light = a.base_zero + zero_blocks<kFwdBlock>(a.zero);
    const int n_blocks = a.base_light + (a.n_light + kFwdWaves - 1) / kFwdWaves;

    // the last kernel of the forward carries the stop event
    const dim3 grid(n_blocks, batch, n_slices);
    // 4-element lanes: every row slice of F (elements) and of the output
    // (fp32) starts on a 4-element boundary of an aligned buffer
    // (slices of 65..80 channels, or exactly 64)
    const bool aligned = ldo % 4 == 0 && reinterpret_cast<uintptr_t>(F) % (4 * esize) == 0 &&
                         reinterpret_cast<uintptr_t>(out) % 16 == 0;
    const bool vec = aligned && ((nch == 5 && channels % 4 == 0 && slice_c % 4 == 0) ||
                                 (nch == 4 && slice_c == 64 && channels % 64 == 0) ||
                                 (nch == 8 && slice_c == 128 && channels % 128 == 0));
    const bool maxr = reduce == BEVPOOL_MAX;
    hipEvent_t fstop = combine ? nullptr : stop;
    const bool seg = a.n_planes > 1;   // some combos split into row segments: several passes
    if (maxr && seg) launch_forward<true, true>(a, dtype, grid, nch, vec, stream, start, fstop);
    else if (maxr) launch_forward<true, false>(a, dtype, grid, nch, vec, stream, start, fstop);
    else if (seg) launch_forward<false, true>(a, dtype, grid, nch, vec, stream, start, fstop);
    else launch_forward<false, false>(a, dtype, grid, nch, vec, stream, start, fstop);
    BEVPOOL_HIP(hipGetLastError());
    if (combine) {
        CombineArgs ca;
        ca.out = out;
        ca.multi_begin = plan->multi_begin;
        ca.multi_cell = plan->multi_cell;
        ca.multi_rows = plan->multi_rows;
        ca.empty_cells = plan->empty_cells;
        ca.cell_start = plan->cell_start;
        ca.n_multi = plan->n_multi;
        ca.C = channels;
        ca.ldo = int32_t(ldo);
        ca.mean = a.mean;
        ca.o_bytes = uint32_t(o_bytes);
        ca.zero = z;
        ca.zero.zero_begin = plan->n_empty - n_late;
        ca.zero.zero_end = plan->n_empty;
        ca.n_zblocks = zero_blocks<kBlock>(ca.zero);
        const int n_cblocks = (plan->n_multi + kCombineGroups - 1) / kCombineGroups;
        const dim3 cgrid(ca.n_zblocks + n_cblocks, batch);
        // 4-element lanes when every 80-channel pass holds 65..80 channels
        // on 16-byte boundaries
        const int tail = channels % (kCombineChunks * 16);
        const bool cvec = channels % 4 == 0 && ldo % 4 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0 &&
                          (tail == 0 || tail > 64);
        if (maxr && cvec) hipExtLaunchKernelGGL((k_combine<true, true>), cgrid, dim3(kBlock), 0, stream, nullptr, stop, 0, ca);
        else if (maxr) hipExtLaunchKernelGGL((k_combine<true, false>), cgrid, dim3(kBlock), 0, stream, nullptr, stop, 0, ca);
        else if (cvec) hipExtLaunchKernelGGL((k_combine<false, true>), cgrid, dim3(kBlock), 0, stream, nullptr, stop, 0, ca);
        else hipExtLaunchKernelGGL((k_combine<false, false>), cgrid, dim3(kBlock), 0, stream, nullptr, stop, 0, ca);
        BEVPOOL_HIP(hipGetLastError());
    }
    return BEVPOOL_OK;
}
