// Per-frame BEV pooling: fused lift (depth probability x feature) and
// per-cell sum (BEVFusion, arXiv 2205.13542, Sec. III-B, first paragraph and
// "Interval Reduction"). The paper gives each cell one GPU thread. Here a
// workgroup owns a tile of cells along a bundle of camera rays (from the
// plan), and lanes run across channels.
//
// One persistent workgroup of 8 waves per CU walks its run of tiles as a
// software pipeline. While tile k is reduced from LDS, the loads for tile
// k+1 (its distinct feature rows and depth probabilities) and tile k+2 (its
// point records, cell list and row pixels) are in flight into registers.
// After the reduction, tile k+1 is written into LDS. A tile's reduction:
//   - its points are split into G equal contiguous chunks, one per lane
//     group (L lanes x NCH chunks of CH channels);
//   - each group walks its chunk cell by cell, reading feature slices from
//     LDS (one staged copy per distinct row of the tile) and accumulating
//     P * F in fp32 registers;
//   - a cell that lies wholly inside one chunk is stored at once. Cells cut
//     by chunk edges leave partial sums in LDS, and the chunk holding the
//     cell's start adds them in chunk order and stores the row.
// A tile whose rows do not fit in LDS reads its features from memory
// instead. A single cell with more points than a tile may stage has an
// extra workgroup of its own, which stages it in rounds. Each workgroup
// also zeroes its share of the cells without points.
//
// Every output row is written exactly once, with plain stores. The
// summation order depends only on the plan, so results are deterministic.
// There is no MFMA: this is a gather and a sum, not a contraction.
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace bevpool {
namespace {

// Input access per dtype and chunk width CH (4 elements, or 1 on the
// unaligned path), widened exactly to fp32.
template <int DT, int CH>
struct In;

template <>
struct In<BEVPOOL_F32, 4> {
    using T = float;
    using Raw = uint4;
    static __device__ __forceinline__ void widen(const Raw &r, float *f) {
        f[0] = __uint_as_float(r.x);
        f[1] = __uint_as_float(r.y);
        f[2] = __uint_as_float(r.z);
        f[3] = __uint_as_float(r.w);
    }
};

template <>
struct In<BEVPOOL_BF16, 4> {
    using T = uint16_t;
    using Raw = uint2;
    static __device__ __forceinline__ void widen(const Raw &r, float *f) {
        f[0] = __uint_as_float(r.x << 16);
        f[1] = __uint_as_float(r.x & 0xFFFF0000u);
        f[2] = __uint_as_float(r.y << 16);
        f[3] = __uint_as_float(r.y & 0xFFFF0000u);
    }
};

template <>
struct In<BEVPOOL_F16, 4> {
    using T = _Float16;
    using Raw = uint2;
    typedef _Float16 half4 __attribute__((ext_vector_type(4)));
    static __device__ __forceinline__ void widen(const Raw &r, float *f) {
        const half4 h = __builtin_bit_cast(half4, r);
        f[0] = float(h.x);
        f[1] = float(h.y);
        f[2] = float(h.z);
        f[3] = float(h.w);
    }
};

__device__ __forceinline__ float widen1(const float &v) { return v; }
__device__ __forceinline__ float widen1(const uint16_t &v) { return __uint_as_float(uint32_t(v) << 16); }
__device__ __forceinline__ float widen1(const _Float16 &v) { return float(v); }

template <int DT>
struct In<DT, 1> {
    using T = typename In<DT, 4>::T;
    using Raw = T;
    static __device__ __forceinline__ void widen(const Raw &r, float *f) { f[0] = widen1(r); }
};

template <int DT>
__device__ __forceinline__ float load_scalar(const typename In<DT, 4>::T *p) {
    return widen1(*p);
}

template <int DT, int CH>
__device__ __forceinline__ typename In<DT, CH>::Raw load_raw(const typename In<DT, CH>::T *p) {
    return *reinterpret_cast<const typename In<DT, CH>::Raw *>(p);
}

// fp32 accumulator of one lane: NCH chunks of CH channels
template <int CH, int NCH>
struct Acc {
    float v[CH * NCH];
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int k = 0; k < CH * NCH; ++k) v[k] = 0.f;
    }
    __device__ __forceinline__ void add(const float *s) {
#pragma unroll
        for (int k = 0; k < CH * NCH; ++k) v[k] += s[k];
    }
};

struct FwdArgs {
    const void *P;   // [B][n_points]
    const void *F;   // [B][n_pix][C]
    float *out;      // [B][n_cells][C]
    const int32_t *tile_hdr, *tile_cells, *comp_cell_start, *comp_point, *comp_row, *row_pix;
    const int32_t *empty_cells, *heavy_tiles, *group_tile_begin;
    int32_t batch, C, n_cells, n_points, n_pix, n_tiles, n_empty, n_heavy;
    FastDiv div_cpr;  // division by chunks per row, ceil(C / CH)
};

constexpr int kThreads = kPersistentBlock;                    // 512
constexpr int kUnroll = 8;
constexpr int kRecPerThread = kPointBudget / kThreads;        // 4
constexpr int kFChunkPerThread = 8;
constexpr int kFChunks = kFChunkPerThread * kThreads;         // feature chunks a tile may stage
static_assert(kPointBudget % kThreads == 0, "records split evenly over the threads");
static_assert(kMaxTileCells + 1 <= kThreads, "one cell entry per thread");

// Lane groups: L lanes per group, S groups per wave, G per workgroup.
struct Groups {
    int L, S, G, sg, lsg, g;
    bool in_group;
    __device__ __forceinline__ Groups(int lanes, int tid, int waves) {
        L = lanes;
        S = kWaveSize / L;
        G = waves * S;
        const int lane = tid % kWaveSize, wave = tid / kWaveSize;
        sg = lane / L;
        lsg = lane - sg * L;
        in_group = sg < S;
        g = wave * S + sg;
    }
};

// Sum P * F over records [lo, hi) into acc. LDS mode: rec.x is the byte
// offset of the point's row in s_F (which the caller has advanced to the
// channel block); global mode: rec.x is its pixel. Lane lsg reads chunks
// lsg and lsg + L, so each read of a group covers one contiguous run.
template <int DT, int CH, int NCH, bool LDS>
__device__ __forceinline__ void gather_sum(const unsigned char *s_F, const typename In<DT, CH>::T *Fc,
                                           int C, int Crem, int L, int lsg, const int2 *s_rec,
                                           int lo, int hi, Acc<CH, NCH> &acc) {
    using R = typename In<DT, CH>::Raw;
    using T = typename In<DT, CH>::T;
    // element offset of each chunk in the row; a chunk past the row's end
    // (last, partial channel block) reads the row's first chunk instead,
    // and its sums are never stored
    int goff[NCH];
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
        goff[k] = (lsg + k * L) * CH;
        if (goff[k] >= Crem) goff[k] = 0;
    }
    auto fetch = [&](int2 e, R *r) {
#pragma unroll
        for (int k = 0; k < NCH; ++k) {
            if (LDS) r[k] = *reinterpret_cast<const R *>(s_F + e.x + goff[k] * int(sizeof(T)));
            else r[k] = load_raw<DT, CH>(Fc + int64_t(e.x) * C + goff[k]);
        }
    };
    auto fma_in = [&](float p, const R *r) {
#pragma unroll
        for (int k = 0; k < NCH; ++k) {
            float f[CH];
            In<DT, CH>::widen(r[k], f);
#pragma unroll
            for (int q = 0; q < CH; ++q) acc.v[k * CH + q] = fmaf(p, f[q], acc.v[k * CH + q]);
        }
    };
    int i = lo;
    for (; i + kUnroll <= hi; i += kUnroll) {
        int2 e[kUnroll];
        R r[kUnroll][NCH];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) e[u] = s_rec[i + u];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) fetch(e[u], r[u]);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) fma_in(__int_as_float(e[u].y), r[u]);
    }
    for (; i < hi; ++i) {
        const int2 e = s_rec[i];
        R r[NCH];
        fetch(e, r);
        fma_in(__int_as_float(e.y), r);
    }
}

// store a lane's chunks of one output row; Crem = channels left in the row
template <int CH, int NCH>
__device__ __forceinline__ void store_acc(float *row, int Crem, int L, int lsg, const Acc<CH, NCH> &acc) {
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
        const int ch = (lsg + k * L) * CH;
        if (ch < Crem) {
            if (CH == 4) {
                *reinterpret_cast<float4 *>(row + ch) =
                    make_float4(acc.v[k * CH], acc.v[k * CH + 1], acc.v[k * CH + 2], acc.v[k * CH + 3]);
            } else {
                row[ch] = acc.v[k * CH];
            }
        }
    }
}

// partial sums in LDS: slot s holds L lanes x (CH * NCH) floats
template <int CH, int NCH>
__device__ __forceinline__ float *part_slot(float *s_part, int slot, int L, int lsg) {
    return s_part + (slot * L + lsg) * (CH * NCH);
}

// A tile header: cell list, points and staged rows of one work item.
struct Hdr {
    int tcb, ncell, tpb, npts, trb, nrows, frame;
    bool direct;
};

// A header is fetched raw and decoded later: reading its fields at once
// would make the wave wait for every load issued before it.
struct RawHdr {
    int4 x, y;
    int item;
};

__device__ __forceinline__ RawHdr fetch_hdr(const FwdArgs &a, int item, int t_begin, int n_items) {
    RawHdr r{make_int4(0, 0, 0, 0), make_int4(0, 0, 0, 0), item};
    if (item < n_items) {
        // through the scalar cache: the wave does not wait on vector loads
        typedef __attribute__((address_space(4))) const int const_int;
        const int t = t_begin + item / a.batch;
        const const_int *p = (const const_int *)(a.tile_hdr + 8 * int64_t(t));
        r.x = make_int4(p[0], p[1], p[2], p[3]);
        r.y = make_int4(p[4], p[5], p[6], p[7]);
    }
    return r;
}

__device__ __forceinline__ Hdr decode_hdr(const FwdArgs &a, const RawHdr &r, int cpr) {
    Hdr h{0, 0, 0, 0, 0, 0, 0, false};
    h.frame = r.item - (r.item / a.batch) * a.batch;
    if (r.x.w <= kPointBudget) {  // heavier tiles have workgroups of their own
        h.tcb = r.x.x;
        h.ncell = r.x.y;
        h.tpb = r.x.z;
        h.npts = r.x.w;
        h.trb = r.y.x;
        h.nrows = r.y.y;
    }
    h.direct = int64_t(h.nrows) * cpr > kFChunks;
    return h;
}

// Loads of a work item that need only its header: point ids, rows, cell
// entries, and the pixel of every feature chunk this thread will stage.
struct Rec {
    int pid[kRecPerThread], row[kRecPerThread], fpix[kFChunkPerThread], cs, cid;
};

__device__ __forceinline__ void load_records(const FwdArgs &a, const Hdr &h, int cpr, int tid, Rec &r) {
#pragma unroll
    for (int i = 0; i < kRecPerThread; ++i) {
        const int j = tid + i * kThreads;
        r.pid[i] = 0;
        r.row[i] = 0;
        if (j < h.npts) {
            r.pid[i] = a.comp_point[h.tpb + j];
            r.row[i] = a.comp_row[h.tpb + j];
        }
    }
    const int nchunks = h.direct ? 0 : h.nrows * cpr;
#pragma unroll
    for (int i = 0; i < kFChunkPerThread; ++i) {
        const int j = tid + i * kThreads;
        r.fpix[i] = 0;
        if (j < nchunks) r.fpix[i] = a.row_pix[h.trb + int(fdiv(uint32_t(j), a.div_cpr))];
    }
    r.cs = (tid <= h.ncell && h.npts > 0) ? a.comp_cell_start[h.tcb + tid] : 0;
    r.cid = (tid < h.ncell && h.npts > 0) ? a.tile_cells[h.tcb + tid] : 0;
}

// Loads that need the records: feature chunks, depth probabilities and,
// for a tile read from memory, each point's pixel.
template <int DT, int CH>
struct Stage {
    typename In<DT, CH>::Raw v[kFChunkPerThread];
    float pv[kRecPerThread];
    int x[kRecPerThread];
};

template <int DT, int CH>
__device__ __forceinline__ void load_stage(const FwdArgs &a, const Hdr &h, int cpr, int tid,
                                           const Rec &r, Stage<DT, CH> &st) {
    using T = typename In<DT, CH>::T;
    const T *Pb = static_cast<const T *>(a.P) + int64_t(h.frame) * a.n_points;
    const T *Fb = static_cast<const T *>(a.F) + int64_t(h.frame) * a.n_pix * a.C;
    const int nchunks = h.direct ? 0 : h.nrows * cpr;
#pragma unroll
    for (int i = 0; i < kFChunkPerThread; ++i) {
        const int j = tid + i * kThreads;
        if (j < nchunks) {
            const int q = j - int(fdiv(uint32_t(j), a.div_cpr)) * cpr;
            st.v[i] = load_raw<DT, CH>(Fb + int64_t(r.fpix[i]) * a.C + q * CH);
        }
    }
#pragma unroll
    for (int i = 0; i < kRecPerThread; ++i) {
        const int j = tid + i * kThreads;
        st.pv[i] = 0.f;
        st.x[i] = 0;
        if (j < h.npts) {
            st.pv[i] = load_scalar<DT>(Pb + r.pid[i]);
            if (h.direct) st.x[i] = a.row_pix[h.trb + r.row[i]];
        }
    }
}

template <int DT, int CH, int NCH>
__device__ __forceinline__ void reduce_tile(const FwdArgs &a, const Hdr &h, int tid,
                                            unsigned char *s_F, const int2 *s_rec, const int *s_cs,
                                            const int *s_cid, int *s_pcell, float *s_part) {
    using T = typename In<DT, CH>::T;
    using A = Acc<CH, NCH>;
    constexpr int W = CH * NCH;
    const int C = a.C;
    const int npts = h.npts, ncell = h.ncell, tpb = h.tpb;
    if (npts == 0) return;  // uniform across the workgroup
    const T *Fb = static_cast<const T *>(a.F) + int64_t(h.frame) * a.n_pix * C;
    float *ob = a.out + int64_t(h.frame) * a.n_cells * C;
    const Groups gr(min(kWaveSize, (C + W - 1) / W), tid, kPersistentWaves);
    const int cblock = gr.L * W;
    const int ca = npts * gr.g / gr.G, cb = npts * (gr.g + 1) / gr.G;  // this group's chunk

    for (int ch0 = 0; ch0 < C; ch0 += cblock) {
        A head, tail;
        head.zero();
        tail.zero();
        int head_cell = -1, tail_cell = -1;
        const bool lane_live = gr.in_group && ch0 + gr.lsg * CH < C;
        if (gr.in_group && ca < cb) {
            int lo = 0, hi = ncell - 1;  // last j with s_cs[j] - tpb <= ca
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_cs[mid] - tpb <= ca) lo = mid;
                else hi = mid - 1;
            }
            for (int j = lo;; ++j) {
                const int cs = s_cs[j] - tpb, ce = s_cs[j + 1] - tpb;
                A acc;
                acc.zero();
                if (lane_live) {
                    if (h.direct)
                        gather_sum<DT, CH, NCH, false>(s_F, Fb + ch0, C, C - ch0, gr.L, gr.lsg, s_rec,
                                                       max(ca, cs), min(cb, ce), acc);
                    else
                        gather_sum<DT, CH, NCH, true>(s_F + ch0 * int(sizeof(T)), Fb, C, C - ch0, gr.L,
                                                      gr.lsg, s_rec, max(ca, cs), min(cb, ce), acc);
                }
                if (cs < ca) {
                    head = acc;
                    head_cell = j;
                } else if (ce > cb) {
                    tail = acc;
                    tail_cell = j;
                } else if (lane_live) {
                    store_acc<CH, NCH>(ob + int64_t(s_cid[j]) * C + ch0, C - ch0, gr.L, gr.lsg, acc);
                }
                if (ce >= cb) break;
            }
        }
        if (gr.in_group) {
            if (gr.lsg == 0) {
                s_pcell[2 * gr.g] = head_cell;
                s_pcell[2 * gr.g + 1] = tail_cell;
            }
            float *hp = part_slot<CH, NCH>(s_part, 2 * gr.g, gr.L, gr.lsg);
            float *tp = part_slot<CH, NCH>(s_part, 2 * gr.g + 1, gr.L, gr.lsg);
#pragma unroll
            for (int k = 0; k < W; ++k) {
                hp[k] = head.v[k];
                tp[k] = tail.v[k];
            }
        }
        __syncthreads();
        // the chunk holding the start of a cut cell adds the later chunks'
        // partial sums of that cell, in chunk order, and stores the row
        if (lane_live) {
            const int j = s_pcell[2 * gr.g + 1];
            if (j >= 0) {
                A sum;
                sum.zero();
                sum.add(part_slot<CH, NCH>(s_part, 2 * gr.g + 1, gr.L, gr.lsg));
                for (int g2 = gr.g + 1; g2 < gr.G; ++g2) {
                    if (npts * g2 / gr.G == npts * (g2 + 1) / gr.G) continue;  // empty chunk
                    if (s_pcell[2 * g2] != j) break;
                    sum.add(part_slot<CH, NCH>(s_part, 2 * g2, gr.L, gr.lsg));
                }
                store_acc<CH, NCH>(ob + int64_t(s_cid[j]) * C + ch0, C - ch0, gr.L, gr.lsg, sum);
            }
        }
        __syncthreads();  // partial slots free for the next channel block
    }
}

// One cell with more points than a tile may stage: rounds of kPointBudget
// points, features read from memory, every group accumulating the cell,
// partials combined in group order.
template <int DT, int CH, int NCH>
__device__ void heavy_cell(const FwdArgs &a, int tile, int tid, int2 *s_rec, float *s_part) {
    using T = typename In<DT, CH>::T;
    using A = Acc<CH, NCH>;
    constexpr int W = CH * NCH;
    const int C = a.C;
    const int *hd = a.tile_hdr + 8 * int64_t(tile);
    const int tcb = hd[0], tpb = hd[2], npts = hd[3], trb = hd[4];
    const int cid = a.tile_cells[tcb];
    const Groups gr(min(kWaveSize, (C + W - 1) / W), tid, kPersistentWaves);
    for (int fb = 0; fb < a.batch; ++fb) {
        const T *Pb = static_cast<const T *>(a.P) + int64_t(fb) * a.n_points;
        const T *Fb = static_cast<const T *>(a.F) + int64_t(fb) * a.n_pix * C;
        float *orow = a.out + (int64_t(fb) * a.n_cells + cid) * C;
        for (int ch0 = 0; ch0 < C; ch0 += gr.L * W) {
            A acc;
            acc.zero();
            for (int r0 = 0; r0 < npts; r0 += kPointBudget) {
                const int nr = min(kPointBudget, npts - r0);
                __syncthreads();
                for (int i = tid; i < nr; i += kThreads) {
                    const int q = tpb + r0 + i;
                    const int pix = a.row_pix[trb + a.comp_row[q]];
                    s_rec[i] = make_int2(pix, __float_as_int(load_scalar<DT>(Pb + a.comp_point[q])));
                }
                __syncthreads();
                if (gr.in_group && ch0 + gr.lsg * CH < C)
                    gather_sum<DT, CH, NCH, false>(nullptr, Fb + ch0, C, C - ch0, gr.L, gr.lsg, s_rec,
                                                   nr * gr.g / gr.G, nr * (gr.g + 1) / gr.G, acc);
            }
            if (gr.in_group) {
                float *slot = part_slot<CH, NCH>(s_part, gr.g, gr.L, gr.lsg);
#pragma unroll
                for (int k = 0; k < W; ++k) slot[k] = acc.v[k];
            }
            __syncthreads();
            if (gr.in_group && gr.g == 0) {
                A sum;
                sum.zero();
                for (int g2 = 0; g2 < gr.G; ++g2) sum.add(part_slot<CH, NCH>(s_part, g2, gr.L, gr.lsg));
                store_acc<CH, NCH>(orow + ch0, C - ch0, gr.L, gr.lsg, sum);
            }
            __syncthreads();
        }
    }
}

__device__ __forceinline__ void wait_all_loads() {
    __builtin_amdgcn_s_waitcnt(0);  // vmcnt, expcnt and lgkmcnt all zero
}

template <int DT, int CH, int NCH>
__global__ __launch_bounds__(kThreads) void k_forward(FwdArgs a) {
    using T = typename In<DT, CH>::T;
    using R = typename In<DT, CH>::Raw;
    constexpr int W = CH * NCH;
    __shared__ __align__(16) unsigned char s_F[kFChunks * CH * sizeof(T)];  // staged rows
    __shared__ int2 s_rec[kPointBudget];                                    // row offset (or pixel), P
    __shared__ int s_cs[kMaxTileCells + 1];                                 // interval table slice
    __shared__ int s_cid[kMaxTileCells];                                    // cell ids
    __shared__ int s_pcell[2 * kThreads];                                   // cut cells per chunk
    __shared__ __align__(16) float s_part[2 * kThreads * W];                // their partial sums

    const int tid = threadIdx.x;
    const int C = a.C;
    if (int(blockIdx.x) >= kPersistentGroups) {
        heavy_cell<DT, CH, NCH>(a, a.heavy_tiles[blockIdx.x - kPersistentGroups], tid, s_rec, s_part);
        return;
    }
    // Workgroups are dealt to the 8 XCDs round-robin. Remap them so that each
    // XCD walks one contiguous run of tiles: neighbouring tiles share feature
    // rows, which then stay in that XCD's L2.
    const int w = (blockIdx.x & 7) * (kPersistentGroups / 8) + (blockIdx.x >> 3);
    const int t_begin = a.group_tile_begin[w], t_end = a.group_tile_begin[w + 1];
    const int n_items = (t_end - t_begin) * a.batch;
    const int cpr = (C + CH - 1) / CH;

    auto write_item = [&](const Hdr &h, const Rec &r, const Stage<DT, CH> &st) {
        const int row_bytes = cpr * CH * int(sizeof(T));
        const int nchunks = h.direct ? 0 : h.nrows * cpr;
#pragma unroll
        for (int i = 0; i < kFChunkPerThread; ++i) {
            const int j = tid + i * kThreads;
            if (j < nchunks) *reinterpret_cast<R *>(s_F + size_t(j) * CH * sizeof(T)) = st.v[i];
        }
#pragma unroll
        for (int i = 0; i < kRecPerThread; ++i) {
            const int j = tid + i * kThreads;
            if (j < h.npts)
                s_rec[j] = make_int2(h.direct ? st.x[i] : r.row[i] * row_bytes, __float_as_int(st.pv[i]));
        }
        if (tid <= h.ncell) s_cs[tid] = r.cs;
        if (tid < h.ncell) s_cid[tid] = r.cid;
    };

    // prologue: item 0 into LDS, item 1's records in registers
    Hdr hC = decode_hdr(a, fetch_hdr(a, 0, t_begin, n_items), cpr);
    Hdr hN = decode_hdr(a, fetch_hdr(a, 1, t_begin, n_items), cpr);
    Hdr hNN = decode_hdr(a, fetch_hdr(a, 2, t_begin, n_items), cpr);
    Rec rN, rNN;
    Stage<DT, CH> st;
    load_records(a, hC, cpr, tid, rN);
    wait_all_loads();
    load_stage<DT, CH>(a, hC, cpr, tid, rN, st);
    {
        // this workgroup's share of the cells without points
        const int z0 = int(int64_t(a.n_empty) * w / kPersistentGroups);
        const int z1 = int(int64_t(a.n_empty) * (w + 1) / kPersistentGroups);
        const int n = (z1 - z0) * cpr;
        for (int fb = 0; fb < a.batch; ++fb) {
            float *ob = a.out + int64_t(fb) * a.n_cells * C;
            for (int idx = tid; idx < n; idx += kThreads) {
                const int cl = int(fdiv(uint32_t(idx), a.div_cpr));
                const int ch = (idx - cl * cpr) * CH;
                float *row = ob + int64_t(a.empty_cells[z0 + cl]) * C;
                if (CH == 4) *reinterpret_cast<float4 *>(row + ch) = make_float4(0.f, 0.f, 0.f, 0.f);
                else row[ch] = 0.f;
            }
        }
    }
    wait_all_loads();
    write_item(hC, rN, st);
    load_records(a, hN, cpr, tid, rN);
    wait_all_loads();
    __syncthreads();

    for (int k = 0; k < n_items; ++k) {
        // in flight during the reduction of item k: item k+3's header, item
        // k+1's features and probabilities, item k+2's records
        const RawHdr rawF = fetch_hdr(a, k + 3, t_begin, n_items);
        load_stage<DT, CH>(a, hN, cpr, tid, rN, st);
        load_records(a, hNN, cpr, tid, rNN);
        reduce_tile<DT, CH, NCH>(a, hC, tid, s_F, s_rec, s_cs, s_cid, s_pcell, s_part);
        wait_all_loads();
        __syncthreads();  // item k is no longer read from LDS
        write_item(hN, rN, st);
        __syncthreads();
        hC = hN;
        hN = hNN;
        hNN = decode_hdr(a, rawF, cpr);
        rN = rNN;
    }
}

template <int DT, int CH, int NCH>
void launch(const FwdArgs &a, int grid, hipStream_t stream) {
    hipLaunchKernelGGL((k_forward<DT, CH, NCH>), dim3(grid), dim3(kThreads), 0, stream, a);
}

template <int DT>
void launch_dtype(const FwdArgs &a, int grid, int mode, hipStream_t stream) {
    if (mode == 2) launch<DT, 4, 2>(a, grid, stream);
    else if (mode == 1) launch<DT, 4, 1>(a, grid, stream);
    else launch<DT, 1, 1>(a, grid, stream);
}

}  // namespace
}  // namespace bevpool

using namespace bevpool;

int bevpool_launch_forward(const void *P, const void *F, const bevpool_plan_s *plan, float *out,
                           int32_t batch, int32_t channels, int32_t dtype, hipStream_t stream) {
    const bevpool_geometry &g = plan->geom;
    const int64_t n_pix = int64_t(g.n_cams) * g.feat_h * g.feat_w;
    if (n_pix * channels > INT32_MAX || int64_t(plan->n_cells) * channels > INT32_MAX)
        return bevpool_fail(BEVPOOL_ERR_OVERFLOW,
                            "channels=%d: pixel or cell rows exceed int32 element offsets", channels);

    const size_t elem = dtype == BEVPOOL_F32 ? 4 : 2;
    const bool aligned = channels % 4 == 0 && (reinterpret_cast<uintptr_t>(F) % (4 * elem)) == 0 &&
                         (reinterpret_cast<uintptr_t>(out) % 16) == 0;
    // 8 channels per lane when the row splits into whole 8-channel lanes
    const int mode = !aligned ? 0 : (channels % 8 == 0 ? 2 : 1);
    const int chunk = aligned ? 4 : 1;

    FwdArgs a;
    a.P = P;
    a.F = F;
    a.out = out;
    a.tile_hdr = plan->tile_hdr;
    a.tile_cells = plan->tile_cells;
    a.comp_cell_start = plan->comp_cell_start;
    a.comp_point = plan->comp_point;
    a.comp_row = plan->comp_row;
    a.row_pix = plan->row_pix;
    a.empty_cells = plan->empty_cells;
    a.heavy_tiles = plan->heavy_tiles;
    a.group_tile_begin = plan->group_tile_begin;
    a.batch = batch;
    a.C = channels;
    a.n_cells = plan->n_cells;
    a.n_points = int32_t(plan->n_points);
    a.n_pix = int32_t(n_pix);
    a.n_tiles = plan->n_tiles;
    a.n_empty = plan->n_empty;
    a.n_heavy = plan->n_heavy;
    a.div_cpr = make_fastdiv(uint32_t((channels + chunk - 1) / chunk));

    const int grid = kPersistentGroups + plan->n_heavy;
    switch (dtype) {
        case BEVPOOL_F32: launch_dtype<BEVPOOL_F32>(a, grid, mode, stream); break;
        case BEVPOOL_BF16: launch_dtype<BEVPOOL_BF16>(a, grid, mode, stream); break;
        default: launch_dtype<BEVPOOL_F16>(a, grid, mode, stream); break;
    }
    BEVPOOL_HIP(hipGetLastError());
    return BEVPOOL_OK;
}
