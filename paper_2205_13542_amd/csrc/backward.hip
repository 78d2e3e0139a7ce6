// Gradients of the per-frame BEV pooling (BEVFusion, arXiv 2205.13542,
// Sec. III-B: the pooling is one layer of a model trained end to end). The
// pooling is bilinear in (P, F); for G = d loss / d out:
//   dP[b][p]      = F[b][pixel(p)] . G[b][cell(p)]   for a kept point p, else 0
//   dF[b][pixel]  = sum over the kept points p of the pixel of P[b][p] G[b][cell(p)]
//
// Two kernels share the work by blocks of kBwdBlockCols pixel columns of one
// camera (the plan flags the blocks that hold a combo that is not clean).
//
// Clean blocks (every combo's kept rows in one cell, one row range): per
// pixel column w the gradients are two small matrix products over the
// column's gradient rows G_w[d] = G[cell(n, d, w)],
//   dF_w[h][c] = sum_d M[d][h] P[d][h] G_w[d][c]
//   dP_w[d][h] = M[d][h] (sum_c G_w[d][c] F_w[h][c])
// with M the kept-row mask of the combos. k_backward_mma runs both on the
// matrix cores (v_mfma_f32_16x16x4f32, fp32 in and out): a workgroup owns
// two adjacent columns and 16 rows of one camera, its four waves take
// consecutive parts of the depth bins, 16 bins per step. The second product
// takes the channels as its K dimension in the order 16t + 4q + e (t the
// step group, q the lane quarter, e the element), so that F and G arrive as
// 16-byte quads; the first takes the depth bins as K and reads the step's
// gradient rows back transposed from the wave's own LDS copy. The waves' dF
// sums are added in LDS in wave order; every dP element comes from one wave.
// The combos come from the plan's table by column (consecutive depth bins
// adjacent: one 8-byte read per lane covers 64 bins), and P and dP of the
// column pair move as 8-byte pieces (W even; odd widths take the per-row
// kernel).
//
// Other blocks (k_backward): pixel-stationary work on the vector ALUs. A
// workgroup owns kBCols pixel columns x kBRows rows of one camera, and its
// kBWaves waves take consecutive parts of the depth bins. A group of 16
// lanes owns one column; lane j holds the row slice channels (the forward's
// lane layout) of the kBRows feature rows, read once, and the kBRows rows'
// dF sums. For each depth bin the group reads one gradient row when the
// combo (camera, depth bin, column) is clean, or one per kept row otherwise.
// dF gets P x G; dP gets the dot product F . G, reduced across the 16 lanes
// by a transpose-reduce (8 shuffles for the 8 rows' sums). A wave parks the
// dP values of a chunk of depth bins in LDS and writes them after the chunk
// (vector loads and stores share one in-order counter, so a store inside the
// loop would hold up the waits for the next loads). The waves' dF sums are
// added in LDS in wave order and stored once.
//
// Nothing is accumulated with atomics, so repeated calls give bitwise equal
// results. Channel slices run as successive launches; slices after the first
// add their dot products to dP.
#include <stdint.h>

#include <algorithm>

#include "device.h"
#include "internal.h"

namespace bevpool {
namespace {

constexpr int kBRows = 8;                      // pixel rows per lane group
constexpr int kBCols = 4;                      // pixel columns per workgroup (lane groups of a wave)
static_assert(kBwdBlockCols % kBCols == 0, "a workgroup's columns lie in one backward block");
constexpr int kBWaves = 4;                     // depth parts per workgroup
constexpr int kBBlock = kBWaves * kWaveSize;
constexpr int kBStages = 4;                    // depth bins in flight per wave
constexpr int kBChunk = 32;                    // combo cells held in registers per pass (2 per lane)

struct BwdArgs {
    const char *P, *F;
    const float *G;
    float *dP, *dF;
    const int32_t *cop, *combo_cells;
    int32_t N, D, H, W, HW, C, c0, cn;         // channel slice [c0, c0 + cn)
    uint32_t p_bytes, f_bytes, g_bytes, dp_bytes, df_bytes;   // per frame
    uint32_t cop_bytes, cc_bytes;
    int32_t items_w, items_h;                  // column blocks and row blocks per camera
    int32_t part;                              // depth bins per wave
    int32_t accumulate_dp, want_dp, want_df;
    const int32_t *mixed;                      // per backward block: 1 if a combo is not clean
    int32_t skip_clean;                        // 1: blocks without such combos are left to k_backward_mma
    int32_t blocks_w8;                         // backward blocks per camera
};

// One depth bin of a lane group: its combo's cell, each row's cell (lane j:
// row j & 7), each row's probability, and the clean combo's gradient row.
template <int NCH>
struct BStage {
    int cc, cell;
    float pv;
    Row<NCH> g;
};

// Sum of v[0..7] over the 16 lanes of a group, by halving rounds: after
// them lanes j and j ^ 8 hold the total of row j & 7.
__device__ __forceinline__ float transpose_reduce(const float (&v)[kBRows], int j) {
    float a[4], b[2];
    const bool h2 = (j & 4) != 0, h1 = (j & 2) != 0, h0 = (j & 1) != 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float keep = h2 ? v[4 + i] : v[i], send = h2 ? v[i] : v[4 + i];
        a[i] = keep + __shfl_xor(send, 4, 16);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const float keep = h1 ? a[2 + i] : a[i], send = h1 ? a[i] : a[2 + i];
        b[i] = keep + __shfl_xor(send, 2, 16);
    }
    const float keep = h0 ? b[1] : b[0], send = h0 ? b[0] : b[1];
    const float c = keep + __shfl_xor(send, 1, 16);
    return c + __shfl_xor(c, 8, 16);
}

// acc[r] += pv_r * g and dot[r] = f[r] . g for the kBRows rows, pv_r from
// lane r of the group.
template <int R, int NCH>
struct RowTerms {
    static __device__ __forceinline__ void run(float (&acc)[kBRows][NCH], float (&dot)[kBRows],
                                               const Row<NCH> (&f)[kBRows], const Row<NCH> &g,
                                               float pv) {
        const float p = row_bcast<R>(pv);
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < NCH; ++k) {
            acc[R][k] = __builtin_fmaf(p, g.v[k], acc[R][k]);
            s = __builtin_fmaf(f[R].v[k], g.v[k], s);
        }
        dot[R] = s;
        RowTerms<R + 1, NCH>::run(acc, dot, f, g, pv);
    }
};
template <int NCH>
struct RowTerms<kBRows, NCH> {
    static __device__ __forceinline__ void run(float (&)[kBRows][NCH], float (&)[kBRows],
                                               const Row<NCH> (&)[kBRows], const Row<NCH> &, float) {}
};

// The same for a combo that is not clean: row R reads the gradient row of
// its own cell (lane R's cell of the group), if it has one. The rows' loads
// are issued kBEach at a time before their terms, so that one round trip
// serves them (loading and using each row in turn made every row wait for
// all loads in flight).
constexpr int kBEach = 4;
template <int R0, int U, int NCH, bool VEC>
__device__ __forceinline__ void each_loads(Row<NCH> (&g)[kBEach], Rsrc G, uint32_t g_ch, int C, int cell) {
    if constexpr (U < kBEach) {
        const int c = row_bcast<R0 + U>(cell);
        const uint32_t addr = uint32_t(max(c, 0)) * uint32_t(C) * 4u + g_ch;
        load_row<BEVPOOL_F32, NCH, VEC>(g[U], G, c >= 0 ? addr : kOff);
        each_loads<R0, U + 1, NCH, VEC>(g, G, g_ch, C, cell);
    }
}
template <int R0, int U, int NCH>
__device__ __forceinline__ void each_terms(float (&acc)[kBRows][NCH], float (&dot)[kBRows],
                                           const Row<NCH> (&f)[kBRows], const Row<NCH> (&g)[kBEach],
                                           float pv) {
    if constexpr (U < kBEach) {
        constexpr int R = R0 + U;
        const float p = row_bcast<R>(pv);
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < NCH; ++k) {
            acc[R][k] = __builtin_fmaf(p, g[U].v[k], acc[R][k]);
            s = __builtin_fmaf(f[R].v[k], g[U].v[k], s);
        }
        dot[R] = s;
        each_terms<R0, U + 1, NCH>(acc, dot, f, g, pv);
    }
}
template <int R0, int NCH, bool VEC>
__device__ __forceinline__ void row_terms_each(float (&acc)[kBRows][NCH], float (&dot)[kBRows],
                                               const Row<NCH> (&f)[kBRows], Rsrc G, uint32_t g_ch,
                                               int C, int cell, float pv) {
    if constexpr (R0 < kBRows) {
        Row<NCH> g[kBEach];
        each_loads<R0, 0, NCH, VEC>(g, G, g_ch, C, cell);
        each_terms<R0, 0, NCH>(acc, dot, f, g, pv);
        row_terms_each<R0 + kBEach, NCH, VEC>(acc, dot, f, G, g_ch, C, cell, pv);
    }
}

template <int NCH>
constexpr int bwd_stride() { return kBRows * NCH * 16 + 16; }   // one lane group's dF sums in LDS

template <int DT, int NCH, bool VEC>
__global__ __launch_bounds__(kBBlock) void k_backward(BwdArgs a) {
    __shared__ float s_df[(kBWaves - 1) * kBCols * bwd_stride<NCH>()];
    // dP of a chunk: [wave][depth bin of the chunk][row][column]
    __shared__ float s_dp[kBWaves * kBChunk * kBRows * kBCols];
    constexpr uint32_t ES = Elem<DT>::kBytes;
    const int b = blockIdx.y;
    // the row blocks of one column block share its gradient rows: placed on
    // one XCD, two at a time on one CU
    const int item = xcd_cu_remap<2>(blockIdx.x, gridDim.x);
    const int rb = item % a.items_h;
    const int t = item / a.items_h;
    const int cb = t % a.items_w, n = t / a.items_w;
    if (a.skip_clean && a.mixed[n * a.blocks_w8 + cb * kBCols / kBwdBlockCols] == 0) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int j = lane & 15, grp = lane >> 4;
    const int w = cb * kBCols + grp;
    const int h0 = rb * kBRows;
    const int jr = j & 7;                      // this lane's row for indices and probabilities
    const bool in_w = w < a.W;
    const bool row_ok = in_w && h0 + jr < a.H;
    const bool tail_ok = j + 16 * (NCH - 1) < a.cn;

    const Rsrc P = make_rsrc(a.P + int64_t(b) * a.p_bytes, a.p_bytes);
    const Rsrc F = make_rsrc(a.F + int64_t(b) * a.f_bytes, a.f_bytes);
    const Rsrc G = make_rsrc(reinterpret_cast<const char *>(a.G) + int64_t(b) * a.g_bytes, a.g_bytes);
    const Rsrc dP = make_rsrc(reinterpret_cast<const char *>(a.dP) + int64_t(b) * a.dp_bytes, a.dp_bytes);
    const Rsrc dF = make_rsrc(reinterpret_cast<const char *>(a.dF) + int64_t(b) * a.df_bytes, a.df_bytes);
    const Rsrc cop = make_rsrc(a.cop, a.cop_bytes);
    const Rsrc ccs = make_rsrc(a.combo_cells, a.cc_bytes);

    // the group's feature rows, once
    Row<NCH> f[kBRows];
    const uint32_t f_row = uint32_t(a.W) * uint32_t(a.C) * ES;
    const uint32_t f_col = in_w ? (uint32_t(n * a.HW + h0 * a.W + w) * uint32_t(a.C) + uint32_t(a.c0)) * ES : kOff;
#pragma unroll
    for (int r = 0; r < kBRows; ++r) {
        load_row<DT, NCH, VEC>(f[r], F, h0 + r < a.H ? f_col + uint32_t(r) * f_row : kOff);
        // the last value of a tail lane lies past the slice: it must not
        // enter the dot products
        if (!tail_ok) f[r].v[NCH - 1] = 0.f;
    }

    float acc[kBRows][NCH];
#pragma unroll
    for (int r = 0; r < kBRows; ++r)
#pragma unroll
        for (int k = 0; k < NCH; ++k) acc[r][k] = 0.f;

    const uint32_t g_ch = uint32_t(a.c0) * 4u;
    const uint32_t gC = uint32_t(a.C) * 4u;
    const int d_lo = min(a.D, wave * a.part), d_hi = min(a.D, d_lo + a.part);
    // point id of (n, d, h0 + jr, w) is pt0 + d * HW
    const uint32_t pt0 = uint32_t((n * a.D) * a.HW + (h0 + jr) * a.W + w);

    for (int dc = d_lo; dc < d_hi; dc += kBChunk) {
        // the combo cells of this chunk's depth bins: lane j holds bins dc + j and dc + 16 + j
        const int dn = min(kBChunk, d_hi - dc);
        const uint32_t cc_base = uint32_t((n * a.D + dc) * a.W + w) * 4u;
        const int cc_a = in_w && j < dn ? int(__builtin_amdgcn_raw_buffer_load_b32(ccs, int(cc_base + uint32_t(j * a.W) * 4u), 0, 0)) : -1;
        const int cc_b = in_w && 16 + j < dn ? int(__builtin_amdgcn_raw_buffer_load_b32(ccs, int(cc_base + uint32_t((16 + j) * a.W) * 4u), 0, 0)) : -1;
        auto load_stage = [&](BStage<NCH> &st, int i) {   // depth bin dc + i
            const bool ok = i < dn;
            const int cc_src = i < 16 ? cc_a : cc_b;
            st.cc = ok ? __shfl(cc_src, (lane & 48) | (i & 15), 64) : -1;
            const uint32_t p = pt0 + uint32_t(dc + i) * uint32_t(a.HW);
            st.cell = ok && row_ok ? int(__builtin_amdgcn_raw_buffer_load_b32(cop, int(p * 4u), 0, 0)) : -1;
            st.pv = Elem<DT>::load(P, ok && row_ok ? p * ES : kOff);
            load_row<BEVPOOL_F32, NCH, VEC>(st.g, G, st.cc >= 0 ? uint32_t(st.cc) * gC + g_ch : kOff);
        };
        BStage<NCH> st[kBStages];
#pragma unroll
        for (int u = 0; u < kBStages; ++u) {
            load_stage(st[u], u);
            __builtin_amdgcn_sched_barrier(0);
        }
        for (int i0 = 0; i0 < dn; i0 += kBStages) {
#pragma unroll
            for (int u = 0; u < kBStages; ++u) {
                const int i = i0 + u;
                // a dropped row adds nothing and gets dP = 0
                const bool kept = st[u].cell >= 0;
                const float pv = kept ? st[u].pv : 0.f;
                float dot[kBRows];
                if (st[u].cc >= 0) {
                    RowTerms<0, NCH>::run(acc, dot, f, st[u].g, pv);
                } else if (st[u].cc == -2) {
                    row_terms_each<0, NCH, VEC>(acc, dot, f, G, g_ch, a.C, st[u].cell, pv);
                } else {
#pragma unroll
                    for (int r = 0; r < kBRows; ++r) dot[r] = 0.f;
                }
                if (a.want_dp) {
                    const float s = transpose_reduce(dot, j);
                    if (j < kBRows && i < dn)
                        s_dp[((wave * kBChunk + i) * kBRows + j) * kBCols + grp] = kept ? s : 0.f;
                }
                load_stage(st[u], i + kBStages);
            }
        }
        if (a.want_dp) {
            // the chunk's dP, 4 columns (16 contiguous bytes) per 4 lanes:
            // value q of the wave is column q % 4, row q / 4 % 8, bin q / 32
            __builtin_amdgcn_wave_barrier();
            for (int q = lane; q < dn * kBRows * kBCols; q += kWaveSize) {
                const int qc = q % kBCols, qr = (q / kBCols) % kBRows, qi = q / (kBCols * kBRows);
                const int wq = cb * kBCols + qc, hq = h0 + qr;
                const uint32_t off = wq < a.W && hq < a.H
                    ? uint32_t(((n * a.D + dc + qi) * a.H + hq) * a.W + wq) * 4u : kOff;
                float v = s_dp[(wave * kBChunk + qi) * kBRows * kBCols + q % (kBRows * kBCols)];
                if (a.accumulate_dp) v += __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(dP, int(off), 0, 0));
                store_f32(dP, off, v);
            }
            __builtin_amdgcn_wave_barrier();
        }
    }

    if (!a.want_df) return;
    // waves 1.. park their sums in LDS; wave 0 adds them in wave order
    constexpr int BS = bwd_stride<NCH>();
    if (wave > 0) {
        float *slot = s_df + ((wave - 1) * kBCols + grp) * BS + j;
#pragma unroll
        for (int r = 0; r < kBRows; ++r)
#pragma unroll
            for (int k = 0; k < NCH; ++k) slot[(r * NCH + k) * 16] = acc[r][k];
    }
    __syncthreads();
    if (wave > 0) return;
    for (int v = 1; v < kBWaves; ++v) {
        const float *slot = s_df + ((v - 1) * kBCols + grp) * BS + j;
#pragma unroll
        for (int r = 0; r < kBRows; ++r)
#pragma unroll
            for (int k = 0; k < NCH; ++k) acc[r][k] += slot[(r * NCH + k) * 16];
    }
    const uint32_t df_col = in_w ? (uint32_t(n * a.HW + h0 * a.W + w) * uint32_t(a.C) + uint32_t(a.c0)) * 4u : kOff;
    const uint32_t df_row = uint32_t(a.W) * uint32_t(a.C) * 4u;
#pragma unroll
    for (int r = 0; r < kBRows; ++r)
        store_row<NCH, VEC>(dF, h0 + r < a.H ? df_col + uint32_t(r) * df_row : kOff, acc[r], tail_ok);
}


// ---------------------------------------------------------------- matrix cores

constexpr int kMWaves = 4;                     // depth parts per workgroup
constexpr int kMCols = 2;                      // adjacent pixel columns per workgroup
constexpr int kMRows = 16;                     // pixel rows per workgroup (M of the instruction)
constexpr int kMChunk = 16;                    // depth bins per step (N of the dP product)
constexpr int kMBlock = kMWaves * kWaveSize;
constexpr int kMSlice = 80;                    // channels per launch (a multiple of 16)
static_assert(kBwdBlockCols % kMCols == 0, "a column pair lies in one backward block");

typedef float f4v __attribute__((ext_vector_type(4)));

struct MmaArgs {
    const char *P, *F;
    const float *G;
    float *dP, *dF;
    const int2 *combos;                        // [N][W][D]: {cell, rows} of a clean combo, else {-1, 0}
    const int32_t *mixed;                      // [N][blocks_w]: 1 if a combo of the block is not clean
    int32_t D, H, W, C, c0, cn;                // channel slice [c0, c0 + cn), cn a multiple of 4; W even
    uint32_t p_bytes, f_bytes, g_bytes, dp_bytes, df_bytes, cb_bytes;
    int32_t pairs_w, blocks_h, blocks_w;       // column pairs, row blocks, backward blocks per camera
    int32_t part;                              // depth bins per wave, a multiple of kMChunk
    int32_t accumulate_dp, want_dp, want_df;
};

// LDS row stride (floats) of a step's gradient rows: an odd multiple of 16,
// so that the four rows one transposed read touches fall in distinct banks.
template <int T>
constexpr int mma_stride() { return 16 * (T | 1); }

// Two consecutive elements as fp32.
template <int DT>
__device__ __forceinline__ void load_pair(Rsrc r, uint32_t off, float &x, float &y) {
    if constexpr (DT == BEVPOOL_F32) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, int(off), 0, 0);
        x = __uint_as_float(v[0]);
        y = __uint_as_float(v[1]);
    } else {
        const uint32_t v = __builtin_amdgcn_raw_buffer_load_b32(r, int(off), 0, 0);
        if constexpr (DT == BEVPOOL_BF16) {
            x = __uint_as_float(v << 16);
            y = __uint_as_float(v & 0xFFFF0000u);
        } else {
            x = float(__builtin_bit_cast(_Float16, uint16_t(v & 0xFFFFu)));
            y = float(__builtin_bit_cast(_Float16, uint16_t(v >> 16)));
        }
    }
}

__device__ __forceinline__ bool row_kept(int h, int rg) {
    const int lo = rg & 0xFFFF, hi = rg >> 16;
    return uint32_t(h - lo) < uint32_t(hi - lo);
}

template <int DT, int T>
__global__ __launch_bounds__(kMBlock) __attribute__((amdgpu_waves_per_eu(3)))
void k_backward_mma(MmaArgs a) {
    constexpr int S = mma_stride<T>();
    constexpr int kLds = kMWaves * kMCols * kMChunk * S;
    static_assert((kMWaves - 1) * kMCols * T * 4 * kWaveSize <= kLds, "dF exchange fits the step buffers");
    constexpr int kFq = 4 * T + 1;             // quads per feature row in LDS (odd: no bank conflicts)
    __shared__ __attribute__((aligned(16))) float s_g[kLds];
    __shared__ f4v s_f[kMCols * kMRows * kFq];
    constexpr uint32_t ES = Elem<DT>::kBytes;
    const int b = blockIdx.y;
    // the two row blocks of a column pair share its gradient rows: placed on
    // one CU; neighbouring pairs share P lines: placed on one XCD
    const int item = xcd_cu_remap<2>(blockIdx.x, gridDim.x);
    const int rb = item % a.blocks_h;
    const int tt = item / a.blocks_h;
    const int cp = tt % a.pairs_w, n = tt / a.pairs_w;
    const int w0 = cp * kMCols;
    if (a.mixed[n * a.blocks_w + w0 / kBwdBlockCols] != 0) return;   // left to k_backward
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q = lane >> 4, j = lane & 15;
    const int h0 = rb * kMRows;
    const int hj = h0 + j;
    const bool hj_ok = hj < a.H;

    const Rsrc P = make_rsrc(a.P + int64_t(b) * a.p_bytes, a.p_bytes);
    const Rsrc F = make_rsrc(a.F + int64_t(b) * a.f_bytes, a.f_bytes);
    const Rsrc G = make_rsrc(reinterpret_cast<const char *>(a.G) + int64_t(b) * a.g_bytes, a.g_bytes);
    const Rsrc dP = make_rsrc(reinterpret_cast<const char *>(a.dP) + int64_t(b) * a.dp_bytes, a.dp_bytes);
    const Rsrc dF = make_rsrc(reinterpret_cast<const char *>(a.dF) + int64_t(b) * a.df_bytes, a.df_bytes);
    const Rsrc CB = make_rsrc(a.combos, a.cb_bytes);
    const uint32_t HW = uint32_t(a.H) * uint32_t(a.W);
    const int d_lo = min(a.D, wave * a.part), d_hi = min(a.D, d_lo + a.part);

    // combos of up to 64 depth bins, lane l: bin dsup + l (one 8-byte entry
    // per column, consecutive bins adjacent), issued before everything else
    int ccv[kMCols], rgv[kMCols];
    auto load_combos = [&](int dsup) {
#pragma unroll
        for (int i = 0; i < kMCols; ++i) {
            const int d = dsup + lane;
            const bool ok = d < d_hi;
            const uint32_t addr = (uint32_t(n * a.W + w0 + i) * uint32_t(a.D) + uint32_t(d)) * 8u;
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(CB, int(ok ? addr : kOff), 0, 0);
            ccv[i] = ok ? int(v[0]) : -1;
            rgv[i] = ok ? int(v[1]) : 0;
        }
    };
    load_combos(d_lo);

    // the feature rows of the workgroup's two columns and 16 rows, in LDS:
    // quad 4t + q of row (i, r) holds channels c0 + 16t + 4q .. + 3
    for (int x = threadIdx.x; x < kMCols * kMRows * 4 * T; x += kMBlock) {
        const int qd = x % (4 * T), r = (x / (4 * T)) % kMRows, i = x / (4 * T * kMRows);
        const int h = h0 + r;
        const bool ok = (h < a.H) & (4 * qd < a.cn);
        const uint32_t addr = ((uint32_t(n) * HW + uint32_t(h) * uint32_t(a.W) + uint32_t(w0 + i)) * uint32_t(a.C) +
                               uint32_t(a.c0 + 4 * qd)) * ES;
        float v[4];
        Elem<DT>::load4(F, ok ? addr : kOff, v);
        s_f[(i * kMRows + r) * kFq + qd] = f4v{v[0], v[1], v[2], v[3]};
    }

    // dF sums: lane (q, j), value r holds row h0 + 4q + r, channel c0 + 16t + j
    f4v accf[kMCols][T];
#pragma unroll
    for (int i = 0; i < kMCols; ++i)
#pragma unroll
        for (int t = 0; t < T; ++t) accf[i][t] = f4v{0.f, 0.f, 0.f, 0.f};

    float *sg = s_g + wave * (kMCols * kMChunk * S);

    // Loads of one step (16 depth bins from d0 = dsup + k): the gradient rows
    // of bins d0 + j as 16-byte quads in the channel order of the dP product,
    // and P of bins d0 + 4s + q, row h0 + j (operand A of the dF product).
    struct StepIn {
        f4v g[kMCols][T];
        float p[kMCols][4];
    };
    auto load_step = [&](StepIn &in, int dsup, int k) {
        const int d0 = dsup + k;
#pragma unroll
        for (int i = 0; i < kMCols; ++i) {
            const int cc = __shfl(ccv[i], k + j, kWaveSize);
            const uint32_t row = uint32_t(max(cc, 0)) * uint32_t(a.C) + uint32_t(a.c0 + 4 * q);
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const bool ok = (cc >= 0) & (16 * t + 4 * q < a.cn);
                const uint32_t addr = (row + uint32_t(16 * t)) * 4u;
                const auto v = __builtin_amdgcn_raw_buffer_load_b128(G, int(ok ? addr : kOff), 0, 0);
                in.g[i][t] = f4v{__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                                 __uint_as_float(v[3])};
            }
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int d = d0 + 4 * s + q;
            const bool ok = (d < d_hi) & hj_ok;
            const uint32_t pt = uint32_t(n * a.D + d) * HW + uint32_t(hj) * uint32_t(a.W) + uint32_t(w0);
            load_pair<DT>(P, ok ? pt * ES : kOff, in.p[0][s], in.p[1][s]);
        }
    };

    auto run_step = [&](const StepIn &in, int dsup, int k) {
        const int d0 = dsup + k;
        // dP product: lane (q, j), value r is row h0 + 4q + r, bin d0 + j
        f4v accp[kMCols];
#pragma unroll
        for (int i = 0; i < kMCols; ++i) {
            accp[i] = f4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const f4v f = s_f[(i * kMRows + j) * kFq + 4 * t + q];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    accp[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(f[e], in.g[i][t][e], accp[i], 0, 0, 0);
            }
        }
        // the step's gradient rows into this wave's LDS rows, row j = bin d0 + j
#pragma unroll
        for (int i = 0; i < kMCols; ++i)
#pragma unroll
            for (int t = 0; t < T; ++t)
                *reinterpret_cast<f4v *>(&sg[(i * kMChunk + j) * S + 16 * t + 4 * q]) = in.g[i][t];
        // dF product: operand A masked to the combos' kept rows, operand B
        // (K = bin, N = channel) read back transposed
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int i = 0; i < kMCols; ++i) {
                const int rg = __shfl(rgv[i], k + 4 * s + q, kWaveSize);
                const float pm = row_kept(hj, rg) ? in.p[i][s] : 0.f;
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    const float g = sg[(i * kMChunk + 4 * s + q) * S + 16 * t + j];
                    accf[i][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(pm, g, accf[i][t], 0, 0, 0);
                }
            }
        if (a.want_dp) {
            const int d = d0 + j;
            int rgj[kMCols];
#pragma unroll
            for (int i = 0; i < kMCols; ++i) rgj[i] = __shfl(rgv[i], k + j, kWaveSize);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int h = h0 + 4 * q + r;
                const bool ok = (d < d_hi) & (h < a.H);
                const uint32_t off = ok ? (uint32_t(n * a.D + d) * HW + uint32_t(h) * uint32_t(a.W) + uint32_t(w0)) * 4u
                                        : kOff;
                float v0 = row_kept(h, rgj[0]) ? accp[0][r] : 0.f;
                float v1 = row_kept(h, rgj[1]) ? accp[1][r] : 0.f;
                if (a.accumulate_dp) {
                    const auto o = __builtin_amdgcn_raw_buffer_load_b64(dP, int(off), 0, 0);
                    v0 += __uint_as_float(o[0]);
                    v1 += __uint_as_float(o[1]);
                }
                __builtin_amdgcn_raw_buffer_store_b64(
                    (__attribute__((ext_vector_type(2))) uint32_t){__float_as_uint(v0), __float_as_uint(v1)}, dP,
                    int(off), 0, 0);
            }
        }
        __builtin_amdgcn_wave_barrier();
    };

    __syncthreads();   // the feature rows are in LDS
    // steps of 16 bins
    StepIn in0;
    for (int dsup = d_lo; dsup < d_hi; dsup += kWaveSize) {
        if (dsup > d_lo) load_combos(dsup);
        const int dn = min(kWaveSize, d_hi - dsup);
        for (int k = 0; k < dn; k += kMChunk) {
            load_step(in0, dsup, k);
            run_step(in0, dsup, k);
        }
    }

    if (!a.want_df) return;
    // waves 1.. park their sums in LDS; wave 0 adds them in wave order
    __syncthreads();
    if (wave > 0) {
#pragma unroll
        for (int i = 0; i < kMCols; ++i)
#pragma unroll
            for (int t = 0; t < T; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    s_g[((((wave - 1) * kMCols + i) * T + t) * 4 + r) * kWaveSize + lane] = accf[i][t][r];
    }
    __syncthreads();
    if (wave > 0) return;
    for (int v = 1; v < kMWaves; ++v)
#pragma unroll
        for (int i = 0; i < kMCols; ++i)
#pragma unroll
            for (int t = 0; t < T; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    accf[i][t][r] += s_g[((((v - 1) * kMCols + i) * T + t) * 4 + r) * kWaveSize + lane];
#pragma unroll
    for (int i = 0; i < kMCols; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int h = h0 + 4 * q + r;
            const uint32_t row = (uint32_t(n) * HW + uint32_t(h) * uint32_t(a.W) + uint32_t(w0 + i)) * uint32_t(a.C);
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const bool ok = (h < a.H) & (16 * t + j < a.cn);
                store_f32(dF, ok ? (row + uint32_t(a.c0 + 16 * t + j)) * 4u : kOff, accf[i][t][r]);
            }
        }
}

template <int DT>
void launch_mma(const MmaArgs &a, dim3 grid, int tiles, hipStream_t s) {
    switch (tiles) {
        case 1: hipLaunchKernelGGL((k_backward_mma<DT, 1>), grid, dim3(kMBlock), 0, s, a); break;
        case 2: hipLaunchKernelGGL((k_backward_mma<DT, 2>), grid, dim3(kMBlock), 0, s, a); break;
        case 3: hipLaunchKernelGGL((k_backward_mma<DT, 3>), grid, dim3(kMBlock), 0, s, a); break;
        case 4: hipLaunchKernelGGL((k_backward_mma<DT, 4>), grid, dim3(kMBlock), 0, s, a); break;
        default: hipLaunchKernelGGL((k_backward_mma<DT, 5>), grid, dim3(kMBlock), 0, s, a); break;
    }
}

template <int DT>
void launch_bwd(const BwdArgs &a, dim3 grid, int nch, bool vec, hipStream_t s) {
    switch (nch) {
        case 1: hipLaunchKernelGGL((k_backward<DT, 1, false>), grid, dim3(kBBlock), 0, s, a); break;
        case 2: hipLaunchKernelGGL((k_backward<DT, 2, false>), grid, dim3(kBBlock), 0, s, a); break;
        case 3: hipLaunchKernelGGL((k_backward<DT, 3, false>), grid, dim3(kBBlock), 0, s, a); break;
        case 4: hipLaunchKernelGGL((k_backward<DT, 4, false>), grid, dim3(kBBlock), 0, s, a); break;
        default:
            if (vec) hipLaunchKernelGGL((k_backward<DT, 5, true>), grid, dim3(kBBlock), 0, s, a);
            else hipLaunchKernelGGL((k_backward<DT, 5, false>), grid, dim3(kBBlock), 0, s, a);
            break;
    }
}

}  // namespace
}  // namespace bevpool

using namespace bevpool;

int bevpool_launch_backward(const float *G, const void *P, const void *F,
                            const bevpool_plan_s *plan, float *dP, float *dF, int32_t batch,
                            int32_t channels, int32_t dtype, hipStream_t stream) {
    const bevpool_geometry &g = plan->geom;
    const int64_t n_pix = int64_t(g.n_cams) * g.feat_h * g.feat_w;
    const int64_t esize = dtype == BEVPOOL_F32 ? 4 : 2;
    const int64_t p_bytes = plan->n_points * esize;
    const int64_t f_bytes = n_pix * channels * esize;
    const int64_t g_bytes = int64_t(plan->n_cells) * channels * 4;
    const int64_t dp_bytes = plan->n_points * 4;
    const int64_t df_bytes = n_pix * channels * 4;
    constexpr int64_t kLimit = int64_t(1) << 31;
    if (p_bytes >= kLimit || f_bytes >= kLimit || g_bytes >= kLimit || dp_bytes >= kLimit ||
        df_bytes >= kLimit)
        return bevpool_fail(BEVPOOL_ERR_OVERFLOW,
                            "channels=%d: one frame's gradient or input tensor reaches 2 GiB",
                            channels);
    if (batch > 65535)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "batch=%d exceeds 65535 frames per call", batch);

    // Matrix-core kernel for the blocks whose combos are all clean: feature
    // and gradient rows move as 4-element quads, so channels % 4 == 0 and
    // aligned rows; the per-row kernel takes the other blocks (or all blocks).
    const bool quads = channels % 4 == 0 && reinterpret_cast<uintptr_t>(F) % (4 * esize) == 0 &&
                       reinterpret_cast<uintptr_t>(G) % 16 == 0;
    // (a column pair is read and written as one 8-byte piece: W even)
    const bool run_mma = quads && g.feat_w % 2 == 0 && plan->n_bwd_mixed < plan->n_bwd_blocks;
    const bool run_rows = !run_mma || plan->n_bwd_mixed > 0;
    if (run_mma) {
        MmaArgs m;
        m.P = static_cast<const char *>(P);
        m.F = static_cast<const char *>(F);
        m.G = G;
        m.dP = dP;
        m.dF = dF;
        m.combos = plan->combo_cols;
        m.mixed = plan->bwd_mixed;
        m.D = g.n_depth;
        m.H = g.feat_h;
        m.W = g.feat_w;
        m.C = channels;
        m.p_bytes = uint32_t(p_bytes);
        m.f_bytes = uint32_t(f_bytes);
        m.g_bytes = uint32_t(g_bytes);
        m.dp_bytes = dP ? uint32_t(dp_bytes) : 0u;
        m.df_bytes = dF ? uint32_t(df_bytes) : 0u;
        m.cb_bytes = uint32_t(int64_t(g.n_cams) * g.n_depth * g.feat_w * 8);
        m.pairs_w = g.feat_w / kMCols;
        m.blocks_h = (g.feat_h + kMRows - 1) / kMRows;
        m.blocks_w = (g.feat_w + kBwdBlockCols - 1) / kBwdBlockCols;
        const int part = (g.n_depth + kMWaves - 1) / kMWaves;
        m.part = (part + kMChunk - 1) / kMChunk * kMChunk;
        m.want_dp = dP != nullptr;
        m.want_df = dF != nullptr;
        const dim3 grid(g.n_cams * m.pairs_w * m.blocks_h, batch);
        for (int c0 = 0; c0 < channels; c0 += kMSlice) {
            m.c0 = c0;
            m.cn = std::min(kMSlice, channels - c0);
            m.accumulate_dp = c0 > 0;
            const int tiles = (m.cn + 15) / 16;
            switch (dtype) {
                case BEVPOOL_F32: launch_mma<BEVPOOL_F32>(m, grid, tiles, stream); break;
                case BEVPOOL_BF16: launch_mma<BEVPOOL_BF16>(m, grid, tiles, stream); break;
                default: launch_mma<BEVPOOL_F16>(m, grid, tiles, stream); break;
            }
            BEVPOOL_HIP(hipGetLastError());
        }
    }
    if (!run_rows) return BEVPOOL_OK;

    const int n_slices = (channels + kBwdSliceChannels - 1) / kBwdSliceChannels;
    const int slice_c = (channels + n_slices - 1) / n_slices;
    const int nch = (slice_c + 15) / 16;
    const bool vec = nch == 5 && channels % 4 == 0 && slice_c % 4 == 0 &&
                     reinterpret_cast<uintptr_t>(F) % (4 * esize) == 0 &&
                     reinterpret_cast<uintptr_t>(G) % 16 == 0 &&
                     (dF == nullptr || reinterpret_cast<uintptr_t>(dF) % 16 == 0);

    BwdArgs a;
    a.P = static_cast<const char *>(P);
    a.F = static_cast<const char *>(F);
    a.G = G;
    a.dP = dP;
    a.dF = dF;
    a.cop = plan->cell_of_point;
    a.combo_cells = plan->combo_cells;
    a.N = g.n_cams;
    a.D = g.n_depth;
    a.H = g.feat_h;
    a.W = g.feat_w;
    a.HW = g.feat_h * g.feat_w;
    a.C = channels;
    a.p_bytes = uint32_t(p_bytes);
    a.f_bytes = uint32_t(f_bytes);
    a.g_bytes = uint32_t(g_bytes);
    a.dp_bytes = dP ? uint32_t(dp_bytes) : 0u;
    a.df_bytes = dF ? uint32_t(df_bytes) : 0u;
    a.cop_bytes = uint32_t(plan->n_points * 4);
    a.cc_bytes = uint32_t(int64_t(g.n_cams) * g.n_depth * g.feat_w * 4);
    a.items_w = (g.feat_w + kBCols - 1) / kBCols;
    a.items_h = (g.feat_h + kBRows - 1) / kBRows;
    a.part = (g.n_depth + kBWaves - 1) / kBWaves;
    a.want_dp = dP != nullptr;
    a.want_df = dF != nullptr;
    a.mixed = plan->bwd_mixed;
    a.skip_clean = run_mma ? 1 : 0;
    a.blocks_w8 = (g.feat_w + kBwdBlockCols - 1) / kBwdBlockCols;
    const dim3 grid(g.n_cams * a.items_w * a.items_h, batch);
    for (int s = 0; s < n_slices; ++s) {
        a.c0 = s * slice_c;
        a.cn = std::min(slice_c, channels - a.c0);
        a.accumulate_dp = s > 0;
        switch (dtype) {
            case BEVPOOL_F32: launch_bwd<BEVPOOL_F32>(a, grid, nch, vec, stream); break;
            case BEVPOOL_BF16: launch_bwd<BEVPOOL_BF16>(a, grid, nch, vec, stream); break;
            default: launch_bwd<BEVPOOL_F16>(a, grid, nch, vec, stream); break;
        }
        BEVPOOL_HIP(hipGetLastError());
    }
    return BEVPOOL_OK;
}
