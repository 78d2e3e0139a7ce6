// Measurement probe, not part of the pooling library: the time a plain
// streaming kernel takes to move the forward pass's compulsory bytes (read
// the inputs once, write the BEV map once) on this device, and the time of
// an empty launch of the same shape. bench.py --floor reports both beside the
// forward pass, timed the same way (dispatch-attached events, cold caches).
//
// bevpool_floor(in, in_bytes, out, out_bytes, mode, stream, start, stop):
//   mode 0: empty kernel; 1: read in_bytes only; 2: write out_bytes only;
//   3: read in_bytes and write out_bytes. Sizes are multiples of 16 bytes
//   below 2^31; out is required in every mode (at least 16 bytes). Each
//   workgroup streams one contiguous share of each buffer with 16-byte
//   accesses. Returns 0, or -1 on a bad argument or HIP error.
#include <stdint.h>

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

namespace {

using Rsrc = __amdgpu_buffer_rsrc_t;
typedef uint32_t u4v __attribute__((ext_vector_type(4)));
constexpr int kBlock = 256;
constexpr int kUnroll = 8;

__device__ __forceinline__ Rsrc rsrc(const void *p, uint32_t n) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, int(n), 0x00020000);
}

__global__ __launch_bounds__(kBlock) void k_floor(const void *in, uint32_t in_bytes, void *out,
                                                  uint32_t out_bytes, int mode, float *sink) {
    const uint32_t G = gridDim.x, g = blockIdx.x, t = threadIdx.x;
    const uint32_t in_units = in_bytes / 16, out_units = out_bytes / 16;
    const uint32_t r0 = uint32_t(uint64_t(in_units) * g / G), r1 = uint32_t(uint64_t(in_units) * (g + 1) / G);
    const uint32_t w0 = uint32_t(uint64_t(out_units) * g / G), w1 = uint32_t(uint64_t(out_units) * (g + 1) / G);
    const Rsrc ri = rsrc(in, in_bytes), ro = rsrc(out, out_bytes);
    u4v acc = {0u, 0u, 0u, 0u};
    if (mode & 1) {
        for (uint32_t u = r0 + t; u < r1; u += kBlock * kUnroll) {
            u4v v[kUnroll];
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) {
                const uint32_t x = u + uint32_t(k) * kBlock;
                v[k] = __builtin_amdgcn_raw_buffer_load_b128(ri, int(x < r1 ? x * 16u : 0x80000000u), 0, 0);
            }
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) acc ^= v[k];
        }
    }
    if (mode & 2) {
        for (uint32_t u = w0 + t; u < w1; u += kBlock)
            __builtin_amdgcn_raw_buffer_store_b128(acc & (u4v){0u, 0u, 0u, 0u}, ro, int(u * 16u), 0, 0);
    }
    if ((mode & 1) && acc[0] == 0x7FC00001u && acc[1] == 0x7FC00002u) sink[0] = 1.f;   // keeps the loads
}

}  // namespace

extern "C" __attribute__((visibility("default"))) int bevpool_floor(
    const void *in, int64_t in_bytes, void *out, int64_t out_bytes, int mode, void *stream,
    void *start, void *stop) {
    if (in_bytes < 0 || out_bytes < 0 || in_bytes % 16 || out_bytes % 16 ||
        in_bytes >= (int64_t(1) << 31) || out_bytes >= (int64_t(1) << 31) || mode < 0 || mode > 3 ||
        ((mode & 1) && !in) || !out || out_bytes < 16)
        return -1;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return -1;
    const dim3 grid(uint32_t(cus > 0 ? cus : 256) * 8);
    hipExtLaunchKernelGGL(k_floor, grid, dim3(kBlock), 0, hipStream_t(stream), hipEvent_t(start),
                          hipEvent_t(stop), 0, in, uint32_t(in_bytes), out, uint32_t(out_bytes), mode,
                          static_cast<float *>(out));
    return hipGetLastError() == hipSuccess ? 0 : -1;
}
