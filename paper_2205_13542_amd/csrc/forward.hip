// Per-frame BEV pooling: fused lift (depth probability x feature) and
// per-cell sum (BEVFusion, arXiv 2205.13542, Sec. III-B, first paragraph and
// "Interval Reduction"). The paper assigns one GPU thread per cell. Here a
// workgroup owns a tile of consecutive cells, and lanes run across channels.
//
// One workgroup (4 waves) per tile of consecutive cells from the plan:
//   1. stage the tile's slice of the interval table in LDS (coalesced);
//   2. stage the tile's points in LDS: pixel index (decoded from the point
//      id) and depth probability (a scattered scalar read per point);
//   3. split the tile's points into G equal contiguous chunks, one per lane
//      group of L = C/4 lanes (3 groups per wave at C = 80). Each group walks
//      its chunk cell by cell, gathering float4 slices of the pixels' feature
//      rows and accumulating P * F in fp32 registers;
//   4. a cell that lies wholly inside one chunk is stored at once. A cell
//      cut by chunk edges leaves partial sums in LDS, and the chunk where
//      the cell starts adds them in chunk order and stores the row;
//   5. cells with no point get zero rows.
// Every output row is written exactly once with plain stores, and the
// summation order depends only on the plan, so results are deterministic.
// The F rows and the output rows are read and written channel-contiguous.
// There is no MFMA: this is a gather and a sum, not a contraction.
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace bevpool {
namespace {

// Input element access per dtype: scalar (depth probability) and 4-wide
// (feature slice) loads, widened exactly to fp32.
template <int DT>
struct In;

template <>
struct In<BEVPOOL_F32> {
    using T = float;
    static __device__ __forceinline__ float one(const T *p) { return *p; }
    static __device__ __forceinline__ float4 four(const T *p) {
        return *reinterpret_cast<const float4 *>(p);
    }
};

template <>
struct In<BEVPOOL_BF16> {
    using T = uint16_t;
    static __device__ __forceinline__ float one(const T *p) {
        return __uint_as_float(uint32_t(*p) << 16);
    }
    static __device__ __forceinline__ float4 four(const T *p) {
        const uint2 v = *reinterpret_cast<const uint2 *>(p);
        return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
                           __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u));
    }
};

template <>
struct In<BEVPOOL_F16> {
    using T = _Float16;
    typedef _Float16 half4 __attribute__((ext_vector_type(4)));
    static __device__ __forceinline__ float one(const T *p) { return float(*p); }
    static __device__ __forceinline__ float4 four(const T *p) {
        const half4 v = *reinterpret_cast<const half4 *>(p);
        return make_float4(float(v.x), float(v.y), float(v.z), float(v.w));
    }
};

// VEC channels per lane: 4 on the aligned fast path, 1 otherwise.
template <int DT, int VEC>
struct Acc;

template <int DT>
struct Acc<DT, 4> {
    float4 v;
    __device__ __forceinline__ void zero() { v = make_float4(0.f, 0.f, 0.f, 0.f); }
    __device__ __forceinline__ void fma(float p, const float4 &f) {
        v.x = fmaf(p, f.x, v.x);
        v.y = fmaf(p, f.y, v.y);
        v.z = fmaf(p, f.z, v.z);
        v.w = fmaf(p, f.w, v.w);
    }
    static __device__ __forceinline__ float4 load(const typename In<DT>::T *p) {
        return In<DT>::four(p);
    }
    static __device__ __forceinline__ float4 vzero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
    __device__ __forceinline__ void add_lds(const float *s) {
        const float4 t = *reinterpret_cast<const float4 *>(s);
        v.x += t.x;
        v.y += t.y;
        v.z += t.z;
        v.w += t.w;
    }
    __device__ __forceinline__ void to_lds(float *s) const { *reinterpret_cast<float4 *>(s) = v; }
    __device__ __forceinline__ void from_lds(const float *s) {
        v = *reinterpret_cast<const float4 *>(s);
    }
    __device__ __forceinline__ void store(float *o) const { *reinterpret_cast<float4 *>(o) = v; }
    static __device__ __forceinline__ void store_zero(float *o) {
        *reinterpret_cast<float4 *>(o) = make_float4(0.f, 0.f, 0.f, 0.f);
    }
};

template <int DT>
struct Acc<DT, 1> {
    float v;
    __device__ __forceinline__ void zero() { v = 0.f; }
    __device__ __forceinline__ void fma(float p, float f) { v = fmaf(p, f, v); }
    static __device__ __forceinline__ float load(const typename In<DT>::T *p) {
        return In<DT>::one(p);
    }
    static __device__ __forceinline__ float vzero() { return 0.f; }
    __device__ __forceinline__ void add_lds(const float *s) { v += *s; }
    __device__ __forceinline__ void to_lds(float *s) const { *s = v; }
    __device__ __forceinline__ void from_lds(const float *s) { v = *s; }
    __device__ __forceinline__ void store(float *o) const { *o = v; }
    static __device__ __forceinline__ void store_zero(float *o) { *o = 0.f; }
};

struct FwdArgs {
    const void *P;   // [B][NP]
    const void *F;   // [B][n_pix][C]
    float *out;      // [B][n_cells][C]
    const int32_t *sorted_point;
    const int32_t *cell_start;
    const int32_t *tile_cell;
    int32_t batch, C, n_cells, n_points, n_pix, HW, n_tiles;
    FastDiv div_dhw, div_hw;
    int32_t L;   // lanes per group
    int32_t S;   // groups per wave
    int32_t CH;  // channels covered by a group in one pass = L * VEC
};

constexpr int kUnroll = 8;

// Sum P * F over staged points [lo, hi) into acc (one group's lanes).
template <int DT, int VEC>
__device__ __forceinline__ void gather_sum(const typename In<DT>::T *Fc, const int2 *s_pt, int lo,
                                           int hi, int C, bool lane_on, Acc<DT, VEC> &acc) {
    using A = Acc<DT, VEC>;
    using V = decltype(A::load(Fc));
    int i = lo;
    for (; i + kUnroll <= hi; i += kUnroll) {
        int2 e[kUnroll];
        V f[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) e[u] = s_pt[i + u];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            f[u] = lane_on ? A::load(Fc + int64_t(e[u].x) * C) : A::vzero();
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) acc.fma(__int_as_float(e[u].y), f[u]);
    }
    for (; i < hi; ++i) {
        const int2 e = s_pt[i];
        const V f = lane_on ? A::load(Fc + int64_t(e.x) * C) : A::vzero();
        acc.fma(__int_as_float(e.y), f);
    }
}

template <int DT, int VEC>
__global__ __launch_bounds__(kBlock) void k_forward(FwdArgs a) {
    using T = typename In<DT>::T;
    using A = Acc<DT, VEC>;
    extern __shared__ __align__(16) unsigned char smem[];
    int2 *s_pt = reinterpret_cast<int2 *>(smem);                    // [kStagePoints]
    int *s_cs = reinterpret_cast<int *>(s_pt + kStagePoints);       // [kMaxTileCells + 1]
    int *s_pcell = s_cs + ((kMaxTileCells + 1 + 3) & ~3);           // [2 * G]
    float *s_pval = reinterpret_cast<float *>(s_pcell + 2 * kBlock); // [2 * G][CH]

    // Consecutive workgroups are spread over the XCDs round-robin; remap so
    // that each XCD walks one contiguous run of tiles (neighbouring cells
    // share feature rows, which then stay in that XCD's L2).
    int tile;
    {
        const int n = a.n_tiles, b = blockIdx.x, xcd = b & 7, per = n >> 3, rem = n & 7;
        tile = xcd * per + (xcd < rem ? xcd : rem) + (b >> 3);
    }
    const int tid = threadIdx.x;
    const int c0 = a.tile_cell[tile];
    const int ncell = a.tile_cell[tile + 1] - c0;
    for (int i = tid; i <= ncell; i += kBlock) s_cs[i] = a.cell_start[c0 + i];
    __syncthreads();
    const int s0 = s_cs[0];
    const int npts = s_cs[ncell] - s0;

    const int wave = tid / kWaveSize, lane = tid % kWaveSize;
    const int sg = lane / a.L, lsg = lane - sg * a.L;
    const bool in_group = sg < a.S;
    const int G = kWaves * a.S;
    const int g = wave * a.S + sg;
    const int C = a.C, CH = a.CH;
    const T *P = static_cast<const T *>(a.P);
    const T *F = static_cast<const T *>(a.F);

    auto pixel_of = [&](int p) -> int {
        const int n = int(fdiv(uint32_t(p), a.div_dhw));
        const int q = int(fdiv(uint32_t(p), a.div_hw));
        return n * a.HW + (p - q * a.HW);
    };

    if (npts > kStagePoints) {
        // a single cell too large to stage at once: rounds of kStagePoints,
        // every group accumulating the same cell, combined in group order
        for (int b = 0; b < a.batch; ++b) {
            const T *Pb = P + int64_t(b) * a.n_points;
            const T *Fb = F + int64_t(b) * a.n_pix * C;
            float *ob = a.out + (int64_t(b) * a.n_cells + c0) * C;
            for (int ch0 = 0; ch0 < C; ch0 += CH) {
                const int choff = ch0 + lsg * VEC;
                const bool lane_on = in_group && choff < C;
                A acc;
                acc.zero();
                for (int r0 = 0; r0 < npts; r0 += kStagePoints) {
                    const int nr = min(kStagePoints, npts - r0);
                    __syncthreads();
                    for (int i = tid; i < nr; i += kBlock) {
                        const int p = a.sorted_point[s0 + r0 + i];
                        s_pt[i] = make_int2(pixel_of(p), __float_as_int(In<DT>::one(Pb + p)));
                    }
                    __syncthreads();
                    if (in_group)
                        gather_sum<DT, VEC>(Fb + choff, s_pt, nr * g / G, nr * (g + 1) / G, C,
                                            lane_on, acc);
                }
                if (lane_on) acc.to_lds(s_pval + g * CH + lsg * VEC);
                __syncthreads();
                if (g == 0 && lane_on) {
                    A sum;
                    sum.from_lds(s_pval + lsg * VEC);
                    for (int g2 = 1; g2 < G; ++g2) sum.add_lds(s_pval + g2 * CH + lsg * VEC);
                    sum.store(ob + choff);
                }
                __syncthreads();
            }
        }
        return;
    }

    // stage the tile's pixel indices once; point ids stay in registers
    int pid[kStagePerThread];
#pragma unroll
    for (int k = 0; k < kStagePerThread; ++k) {
        const int i = tid + k * kBlock;
        pid[k] = 0;
        if (i < npts) {
            pid[k] = a.sorted_point[s0 + i];
            s_pt[i].x = pixel_of(pid[k]);
        }
    }
    const int ca = npts * g / G, cb = npts * (g + 1) / G;  // this group's chunk

    for (int b = 0; b < a.batch; ++b) {
        const T *Pb = P + int64_t(b) * a.n_points;
        const T *Fb = F + int64_t(b) * a.n_pix * C;
        float *ob = a.out + int64_t(b) * a.n_cells * C;
#pragma unroll
        for (int k = 0; k < kStagePerThread; ++k) {
            const int i = tid + k * kBlock;
            if (i < npts) s_pt[i].y = __float_as_int(In<DT>::one(Pb + pid[k]));
        }
        __syncthreads();

        for (int ch0 = 0; ch0 < C; ch0 += CH) {
            const int choff = ch0 + lsg * VEC;
            const bool lane_on = in_group && choff < C;
            if (in_group) {
                s_pcell[2 * g] = -1;
                s_pcell[2 * g + 1] = -1;
            }
            if (in_group && ca < cb) {
                // the cell holding local point ca: last j with s_cs[j] - s0 <= ca
                int lo = 0, hi = ncell - 1;
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (s_cs[mid] - s0 <= ca) lo = mid;
                    else hi = mid - 1;
                }
                int j = lo;
                while (true) {
                    const int cs = s_cs[j] - s0, ce = s_cs[j + 1] - s0;
                    A acc;
                    acc.zero();
                    gather_sum<DT, VEC>(Fb + choff, s_pt, max(ca, cs), min(cb, ce), C, lane_on, acc);
                    if (cs >= ca && ce <= cb) {
                        if (lane_on) acc.store(ob + int64_t(c0 + j) * C + choff);
                    } else {
                        const int slot = 2 * g + (cs < ca ? 0 : 1);
                        if (lsg == 0) s_pcell[slot] = j;
                        if (lane_on) acc.to_lds(s_pval + slot * CH + lsg * VEC);
                    }
                    if (ce >= cb) break;
                    ++j;
                    while (s_cs[j + 1] == s_cs[j]) ++j;  // skip empty cells
                }
            }
            __syncthreads();
            // a chunk holding the start of a cut cell adds the later chunks'
            // partial sums of that cell, in chunk order, and stores the row
            if (in_group) {
                const int j = s_pcell[2 * g + 1];
                if (j >= 0) {
                    A sum;
                    sum.zero();
                    if (lane_on) sum.from_lds(s_pval + (2 * g + 1) * CH + lsg * VEC);
                    for (int g2 = g + 1; g2 < G; ++g2) {
                        if (npts * g2 / G == npts * (g2 + 1) / G) continue;  // empty chunk
                        if (s_pcell[2 * g2] != j) break;
                        if (lane_on) sum.add_lds(s_pval + (2 * g2) * CH + lsg * VEC);
                    }
                    if (lane_on) sum.store(ob + int64_t(c0 + j) * C + choff);
                }
            }
            __syncthreads();
        }
        // cells without points
        if (in_group) {
            for (int cl = g; cl < ncell; cl += G) {
                if (s_cs[cl + 1] != s_cs[cl]) continue;
                float *row = ob + int64_t(c0 + cl) * C;
                for (int ch = lsg * VEC; ch < C; ch += CH) A::store_zero(row + ch);
            }
        }
    }
}

// LDS: staged points, interval-table slice, partial-sum cell ids, and two
// partial-sum rows per group (G groups of CH channels, G * CH <= 4 * 256).
size_t forward_lds_bytes(int groups, int CH) {
    return sizeof(int2) * kStagePoints + sizeof(int) * ((kMaxTileCells + 1 + 3) & ~3) +
           sizeof(int) * 2 * kBlock + sizeof(float) * 2 * size_t(groups) * size_t(CH);
}

template <int DT, int VEC>
int launch(const FwdArgs &a, hipStream_t stream) {
    const size_t lds = forward_lds_bytes(kWaves * a.S, a.CH);
    hipLaunchKernelGGL((k_forward<DT, VEC>), dim3(a.n_tiles), dim3(kBlock), lds, stream, a);
    return BEVPOOL_OK;
}

}  // namespace
}  // namespace bevpool

using namespace bevpool;

int bevpool_launch_forward(const void *P, const void *F, const bevpool_plan_s *plan, float *out,
                           int32_t batch, int32_t channels, int32_t dtype, hipStream_t stream) {
    const bevpool_geometry &g = plan->geom;
    const int64_t hw = int64_t(g.feat_h) * g.feat_w;
    const int64_t n_pix = int64_t(g.n_cams) * hw;
    if (n_pix * channels > INT32_MAX || int64_t(plan->n_cells) * channels > INT32_MAX)
        return bevpool_fail(BEVPOOL_ERR_OVERFLOW,
                            "channels=%d: pixel or cell rows exceed int32 element offsets", channels);

    const size_t elem = dtype == BEVPOOL_F32 ? 4 : 2;
    const bool aligned = channels % 4 == 0 && (reinterpret_cast<uintptr_t>(F) % (4 * elem)) == 0 &&
                         (reinterpret_cast<uintptr_t>(out) % 16) == 0;
    const int VEC = aligned ? 4 : 1;

    FwdArgs a;
    a.P = P;
    a.F = F;
    a.out = out;
    a.sorted_point = plan->sorted_point;
    a.cell_start = plan->cell_start;
    a.tile_cell = plan->tile_cell;
    a.batch = batch;
    a.C = channels;
    a.n_cells = plan->n_cells;
    a.n_points = int32_t(plan->n_points);
    a.n_pix = int32_t(n_pix);
    a.HW = int32_t(hw);
    a.n_tiles = plan->n_tiles;
    a.div_dhw = make_fastdiv(uint32_t(int64_t(g.n_depth) * hw));
    a.div_hw = make_fastdiv(uint32_t(hw));
    const int lanes_needed = (channels + VEC - 1) / VEC;
    a.L = lanes_needed < kWaveSize ? lanes_needed : kWaveSize;
    a.S = kWaveSize / a.L;
    a.CH = a.L * VEC;

    int rc;
    switch (dtype * 2 + (VEC == 4 ? 1 : 0)) {
        case BEVPOOL_F32 * 2 + 1: rc = launch<BEVPOOL_F32, 4>(a, stream); break;
        case BEVPOOL_F32 * 2 + 0: rc = launch<BEVPOOL_F32, 1>(a, stream); break;
        case BEVPOOL_BF16 * 2 + 1: rc = launch<BEVPOOL_BF16, 4>(a, stream); break;
        case BEVPOOL_BF16 * 2 + 0: rc = launch<BEVPOOL_BF16, 1>(a, stream); break;
        case BEVPOOL_F16 * 2 + 1: rc = launch<BEVPOOL_F16, 4>(a, stream); break;
        default: rc = launch<BEVPOOL_F16, 1>(a, stream); break;
    }
    if (rc != BEVPOOL_OK) return rc;
    BEVPOOL_HIP(hipGetLastError());
    return BEVPOOL_OK;
}
