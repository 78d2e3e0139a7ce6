// Channel-major copy of a BEV map: [B][ny*nx][C] rows (channels contiguous,
// as the pooling writes them) to [B][C][ny][nx] planes, the layout a
// convolutional BEV encoder reads (BEVFusion, arXiv 2205.13542, Sec. III-C:
// the fused BEV features go through a convolutional encoder).
//
// A pure data movement, bound by HBM: every element is read once and
// written once. (The concatenation that fuses camera and LiDAR maps is a
// concatenation of channel planes in this layout.) A workgroup moves a tile
// of kTileCells consecutive cells x up to kTileCh channels through LDS: it
// reads the tile's rows (for a contiguous map with C <= kTileCh, one
// stretch of 64 * C floats, in 16-byte loads when aligned), and 64
// consecutive lanes write one plane's 64 cells (256 contiguous bytes). The
// LDS rows are padded by one word so that the column-wise LDS stores fall in
// distinct banks.
#include <stdint.h>

#include "internal.h"

namespace bevpool {
namespace {

constexpr int kTileCells = 64;
constexpr int kTileCh = 128;          // channels per tile at most
constexpr int kLayoutBlock = 256;

struct LayoutArgs {
    const float *in;
    float *out;
    int64_t in_frame, out_frame;      // floats per frame
    int32_t n_cells, C, ldi;
    int32_t tile_ch;                  // channels per tile: min(C, kTileCh)
    int32_t vec;                      // rows read as float4 (aligned, C and ldi multiples of 4)
};

__global__ __launch_bounds__(kLayoutBlock) void k_to_nchw(LayoutArgs a) {
    __shared__ float tile[kTileCh][kTileCells + 1];
    const int cell0 = blockIdx.x * kTileCells;
    const int ch0 = blockIdx.y * a.tile_ch;
    const int tc = min(a.tile_ch, a.C - ch0);         // channels of this tile
    const int nc = min(kTileCells, a.n_cells - cell0);  // cells of this tile
    const float *in = a.in + int64_t(blockIdx.z) * a.in_frame;
    float *out = a.out + int64_t(blockIdx.z) * a.out_frame;
    if (a.vec) {
        // tc / 4 float4 per row; with ldi == C the tile's rows are one
        // contiguous stretch of memory
        const int q = tc >> 2;
        for (int idx = threadIdx.x; idx < nc * q; idx += kLayoutBlock) {
            const int cl = idx / q, c4 = (idx - cl * q) << 2;
            const float4 v = *reinterpret_cast<const float4 *>(in + int64_t(cell0 + cl) * a.ldi + ch0 + c4);
            tile[c4][cl] = v.x;
            tile[c4 + 1][cl] = v.y;
            tile[c4 + 2][cl] = v.z;
            tile[c4 + 3][cl] = v.w;
        }
    } else {
        for (int idx = threadIdx.x; idx < nc * tc; idx += kLayoutBlock) {
            const int cl = idx / tc, ch = idx - cl * tc;
            tile[ch][cl] = in[int64_t(cell0 + cl) * a.ldi + ch0 + ch];
        }
    }
    __syncthreads();
    // 64 consecutive lanes write one plane's cells of the tile
    for (int idx = threadIdx.x; idx < tc * kTileCells; idx += kLayoutBlock) {
        const int ch = idx / kTileCells, cl = idx % kTileCells;
        if (cl < nc) out[int64_t(ch0 + ch) * a.n_cells + cell0 + cl] = tile[ch][cl];
    }
}

}  // namespace
}  // namespace bevpool

using namespace bevpool;

int bevpool_launch_to_nchw(const float *in, int64_t in_row_stride, float *out, int32_t batch,
                           int32_t ny, int32_t nx, int32_t channels, hipStream_t stream) {
    const int64_t n_cells = int64_t(ny) * nx;
    if (in_row_stride >= (int64_t(1) << 31) || n_cells >= (int64_t(1) << 31) - kTileCells)
        return bevpool_fail(BEVPOOL_ERR_OVERFLOW, "ny=%d nx=%d row stride %lld: a cell or channel "
                            "index would not fit in int32", ny, nx, (long long)in_row_stride);
    if (batch > 65535)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "batch=%d exceeds 65535 frames per call", batch);
    LayoutArgs a;
    a.in = in;
    a.out = out;
    a.in_frame = n_cells * in_row_stride;
    a.out_frame = n_cells * channels;
    a.n_cells = int32_t(n_cells);
    a.C = channels;
    a.ldi = int32_t(in_row_stride);
    // tiles of up to kTileCh channels, as even as possible
    const int n_ct = (channels + kTileCh - 1) / kTileCh;
    a.tile_ch = (channels + n_ct - 1) / n_ct;
    a.vec = (a.tile_ch % 4 == 0 && channels % 4 == 0 && in_row_stride % 4 == 0 &&
             reinterpret_cast<uintptr_t>(in) % 16 == 0) ? 1 : 0;
    const dim3 grid(uint32_t((n_cells + kTileCells - 1) / kTileCells), uint32_t(n_ct),
                    uint32_t(batch));
    if (grid.y > 65535)
        return bevpool_fail(BEVPOOL_ERR_INVALID_ARG, "channels=%d: too many channel tiles", channels);
    hipLaunchKernelGGL(k_to_nchw, grid, dim3(kLayoutBlock), 0, stream, a);
    BEVPOOL_HIP(hipGetLastError());
    return BEVPOOL_OK;
}
