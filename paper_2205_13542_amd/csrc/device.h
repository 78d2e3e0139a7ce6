// Device helpers shared by the forward and backward kernels of
// libbevpool.so: raw buffer accesses with out-of-range masking, element
// loads of the three input types, DPP row broadcasts, and the lane layout
// of a row slice across a 16-lane group.
#pragma once

#include <stdint.h>

#include "internal.h"

namespace bevpool {
namespace {

constexpr uint32_t kOff = 0x80000000u;   // past every buffer (sizes stay below 2^31)
constexpr int kRsrcWord3 = 0x00020000;   // gfx9 raw buffer: 32-bit data format

using Rsrc = __amdgpu_buffer_rsrc_t;

__device__ __forceinline__ Rsrc make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, int(bytes), kRsrcWord3);
}

template <int DT>
struct Elem;
// load: one element as fp32; load4: four consecutive elements.
template <>
struct Elem<BEVPOOL_F32> {
    static constexpr uint32_t kBytes = 4;
    static __device__ __forceinline__ float load(Rsrc r, uint32_t off) {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, int(off), 0, 0));
    }
    static __device__ __forceinline__ void load4(Rsrc r, uint32_t off, float *v) {
        const auto q = __builtin_amdgcn_raw_buffer_load_b128(r, int(off), 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = __uint_as_float(q[i]);
    }
};
template <>
struct Elem<BEVPOOL_BF16> {
    static constexpr uint32_t kBytes = 2;
    static __device__ __forceinline__ float load(Rsrc r, uint32_t off) {
        return __uint_as_float(uint32_t(__builtin_amdgcn_raw_buffer_load_b16(r, int(off), 0, 0)) << 16);
    }
    static __device__ __forceinline__ void load4(Rsrc r, uint32_t off, float *v) {
        const auto q = __builtin_amdgcn_raw_buffer_load_b64(r, int(off), 0, 0);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            v[2 * i] = __uint_as_float(uint32_t(q[i]) << 16);
            v[2 * i + 1] = __uint_as_float(uint32_t(q[i]) & 0xFFFF0000u);
        }
    }
};
template <>
struct Elem<BEVPOOL_F16> {
    static constexpr uint32_t kBytes = 2;
    static __device__ __forceinline__ float load(Rsrc r, uint32_t off) {
        return float(__builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(r, int(off), 0, 0)));
    }
    static __device__ __forceinline__ void load4(Rsrc r, uint32_t off, float *v) {
        const auto q = __builtin_amdgcn_raw_buffer_load_b64(r, int(off), 0, 0);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            v[2 * i] = float(__builtin_bit_cast(_Float16, uint16_t(uint32_t(q[i]) & 0xFFFFu)));
            v[2 * i + 1] = float(__builtin_bit_cast(_Float16, uint16_t(uint32_t(q[i]) >> 16)));
        }
    }
};

__device__ __forceinline__ void store_f32(Rsrc r, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, int(off), 0, 0);
}

// Value of lane J of this lane's DPP row (row_newbcast).
template <int J>
__device__ __forceinline__ int row_bcast(int v) {
    return __builtin_amdgcn_mov_dpp(v, 0x150 + J, 0xF, 0xF, false);
}
template <int J>
__device__ __forceinline__ float row_bcast(float v) {
    return __int_as_float(row_bcast<J>(__float_as_int(v)));
}

// Work order for a grid of G workgroups whose consecutive items share
// data. Workgroups are dealt to the 8 XCDs round-robin (block b runs on XCD
// b % 8), so item ranges are given to XCDs in contiguous eighths: adjacent
// items meet in one L2. Within an XCD the dispatcher deals workgroups to
// its 32 CUs in turn, so the XCD's workgroups k, k + 32, ... land on one CU
// while every CU has room (measured on MI355X): the first ROUNDS * 32 of
// them get ROUNDS consecutive items per CU, which then also meet in that
// CU's L1. Placement only affects speed; the map is a permutation of
// 0..G-1 for any G.
constexpr int kCusPerXcd = 32;
template <int ROUNDS>
__device__ __forceinline__ int xcd_cu_remap(int b, int G) {
    const int q = G >> 3, r = G & 7, x = b & 7, k0 = b >> 3;
    constexpr int kSpan = ROUNDS * kCusPerXcd;
    // a permutation of the XCD's first kSpan workgroups (it has >= q)
    const int k = (q >= kSpan && k0 < kSpan) ? ROUNDS * (k0 % kCusPerXcd) + k0 / kCusPerXcd : k0;
    return x < r ? x * (q + 1) + k : r * (q + 1) + (x - r) * q + k;
}

template <int NCH>
struct Row {
    float v[NCH];
};

// Channels of a row slice held by lane j of a 16-lane group: value k is
// channel j + 16k. With VEC (rows starting on 16-byte boundaries), values
// 0..3 are channels 4j..4j+3 instead, so that 64 of the channels move as one
// 4-element access per lane: for slices of 65..80 channels value 4 is
// channel 64 + j (NCH = 5), slices of exactly 64 channels need nothing else
// (NCH = 4), and in slices of exactly 128 values 4..7 are channels
// 64 + 4j..64 + 4j + 3 (NCH = 8). Lanes past the slice's last channel read
// bytes that are never stored.

// Row slice at byte offset off of its first channel (or kOff plus less than
// 2^31: every access is then out of range).
template <int DT, int NCH, bool VEC>
__device__ __forceinline__ void load_row(Row<NCH> &r, Rsrc src, uint32_t off) {
    static_assert(!VEC || NCH == 4 || NCH == 5 || NCH == 8,
                  "4-element lanes hold 64, 65..80 or 128 channels");
    constexpr uint32_t ES = Elem<DT>::kBytes;
    const uint32_t j = threadIdx.x & 15;
    if constexpr (VEC) {
        Elem<DT>::load4(src, off + 4 * j * ES, r.v);
        if constexpr (NCH == 5) r.v[4] = Elem<DT>::load(src, off + (64 + j) * ES);
        if constexpr (NCH == 8) Elem<DT>::load4(src, off + (64 + 4 * j) * ES, r.v + 4);
    } else {
#pragma unroll
        for (int k = 0; k < NCH; ++k) r.v[k] = Elem<DT>::load(src, off + (j + 16 * k) * ES);
    }
}

// Store a row slice of fp32 at byte offset off of its first channel (or
// kOff). Only the last value can lie past the slice: tail_ok says whether it
// does not.
template <int NCH, bool VEC>
__device__ __forceinline__ void store_row(Rsrc dst, uint32_t off, const float *v, bool tail_ok) {
    const uint32_t j = threadIdx.x & 15;
    if constexpr (VEC) {
        // slices of 64 or 128 channels have no tail: all their values are in
        __builtin_amdgcn_raw_buffer_store_b128(
            (__attribute__((ext_vector_type(4))) uint32_t){__float_as_uint(v[0]), __float_as_uint(v[1]),
                                                           __float_as_uint(v[2]), __float_as_uint(v[3])},
            dst, int(NCH == 5 || tail_ok ? off + 16 * j : kOff), 0, 0);
        if constexpr (NCH == 5) store_f32(dst, tail_ok ? off + (64 + j) * 4 : kOff, v[4]);
        if constexpr (NCH == 8)
            __builtin_amdgcn_raw_buffer_store_b128(
                (__attribute__((ext_vector_type(4))) uint32_t){__float_as_uint(v[4]), __float_as_uint(v[5]),
                                                               __float_as_uint(v[6]), __float_as_uint(v[7])},
                dst, int(tail_ok ? off + 256 + 16 * j : kOff), 0, 0);
    } else {
#pragma unroll
        for (int k = 0; k < NCH - 1; ++k) store_f32(dst, off + (j + 16 * k) * 4, v[k]);
        store_f32(dst, tail_ok ? off + (j + 16 * (NCH - 1)) * 4 : kOff, v[NCH - 1]);
    }
}

}  // namespace
}  // namespace bevpool
