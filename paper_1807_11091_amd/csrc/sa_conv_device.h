// Device helpers of the CONV kernels: raw buffer loads that read out-of-range
// offsets as zero, the XCD-aware workgroup order, and the epilogue stores of
// bf16 output tiles staged in LDS.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "sa_device.h"

namespace sa {

constexpr int kRsrcWord3 = 0x00020000;  // raw buffer resource: 32-bit data, range checked
// Offset used for reads that must return zero: every buffer here is smaller
// than 2 GiB, so offset + 16 stays past its range without 32-bit wrap-around.
constexpr uint32_t kInvalidOffset = 0x80000000u;

__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRsrcWord3);
}

__device__ inline uint4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

// Workgroups are dispatched to the 8 XCDs round-robin (id mod 8); each XCD has
// its own L2.  Remap ids so that every XCD walks one contiguous range of tiles
// (neighbouring tiles share input rows and weight slices): XCD x gets the
// range of q+1 tiles when x < r, of q tiles otherwise (n = 8q + r).
__device__ inline int xcd_remap(int bid, int n) {
    const int xcd = bid & 7, local = bid >> 3, q = n >> 3, r = n & 7;
    return xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

// Writes the first min(n, 4) of four consecutive bf16 outputs to the LDS
// output tile at dst with the widest stores dst's alignment allows (output rows
// of any length: a quad is 8-, 4- or 2-byte aligned).
// 16-byte store of output with the non-temporal hint: the output streams past
// the caches instead of evicting the input lines that later tiles re-read
// (measured 3% faster over the compacted and 5% over the dense ResNet-50 CONVs)
__device__ inline void nt_store16(void *p, uint4 v) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(u32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4 *>(p));
}
__device__ inline void stage_quad(uint16_t *dst, const uint16_t *o, int n) {
    const uint32_t lo = o[0] | ((uint32_t)o[1] << 16), hi = o[2] | ((uint32_t)o[3] << 16);
    const uintptr_t ad = reinterpret_cast<uintptr_t>(dst);
    if (n >= 4 && (ad & 7) == 0) {
        *reinterpret_cast<uint2 *>(dst) = make_uint2(lo, hi);
    } else if (n >= 4 && (ad & 3) == 0) {
        reinterpret_cast<uint32_t *>(dst)[0] = lo;
        reinterpret_cast<uint32_t *>(dst)[1] = hi;
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (e < n) dst[e] = o[e];
    }
}

// Stores n <= 8 consecutive bf16 outputs (a 16-byte aligned row of the LDS
// output tile) with the widest stores the destination's alignment allows:
// output rows of sum(M_g) channels are 16-byte aligned only when that sum is a
// multiple of 8 (pruned layers keep any number of filters).
__device__ inline void store_out8(uint16_t *dst, const uint16_t *src, int n) {
    const uintptr_t ad = reinterpret_cast<uintptr_t>(dst);
    if (n == 8 && (ad & 15) == 0) {
        nt_store16(dst, *reinterpret_cast<const uint4 *>(src));
        return;
    }
    if (n == 8 && (ad & 7) == 0) {
        reinterpret_cast<uint2 *>(dst)[0] = reinterpret_cast<const uint2 *>(src)[0];
        reinterpret_cast<uint2 *>(dst)[1] = reinterpret_cast<const uint2 *>(src)[1];
        return;
    }
    int e = 0;
    if (ad & 2) {  // one element to reach 4-byte alignment
        dst[0] = src[0];
        e = 1;
    }
    for (; e + 2 <= n; e += 2)
        *reinterpret_cast<uint32_t *>(dst + e) = (uint32_t)src[e] | ((uint32_t)src[e + 1] << 16);
    if (e < n) dst[e] = src[e];
}

// An output tile that holds whole output rows (one conv group owns every output
// channel and one filter tile covers them) is one contiguous range of Y: it is
// written with 16-byte stores whatever the row length, the elements read back
// from the LDS tile (row pitch RP) one by one.  Y + n0 * Cy is 16-byte aligned
// when Y is (n0 is a multiple of 8).
template <int RP>
__device__ inline void store_tile_rows(uint16_t *Y, const uint16_t *sC, int n0, int rows, int Cy,
                                       const FastDiv &divCy, int tid, int nt) {
    const int total = rows * Cy;
    uint16_t *base = Y + (int64_t)n0 * Cy;
    for (int c = tid; c * 8 < total; c += nt) {
        const int e0 = c * 8;
        int pl = (int)fdiv((uint32_t)e0, divCy);
        int m = e0 - pl * Cy;
        uint16_t v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            v[q] = e0 + q < total ? sC[pl * RP + m] : (uint16_t)0;
            if (++m == Cy) {
                m = 0;
                ++pl;
            }
        }
        if (e0 + 8 <= total) {
            *reinterpret_cast<uint4 *>(base + e0) =
                make_uint4(v[0] | ((uint32_t)v[1] << 16), v[2] | ((uint32_t)v[3] << 16),
                           v[4] | ((uint32_t)v[5] << 16), v[6] | ((uint32_t)v[7] << 16));
        } else {
            for (int q = 0; e0 + q < total; ++q) base[e0 + q] = v[q];
        }
    }
}

// Stores the valid part of a tile row: `count` consecutive bf16 outputs that
// belong at element offset e0 of Y, read from LDS at src[0 .. count).  The
// 8-element (16-byte) chunks are aligned on the addresses of Y (whose start is
// `yshift` elements past a 16-byte boundary), so a row that starts anywhere
// still goes out in whole 16-byte stores except for its first and last chunk,
// which take 2-byte stores of the elements inside the row (the rest of such a
// chunk belongs to a neighbouring tile or row).  Chunk ci of the row: threads
// call this for every ci < (count + 7) / 8 + 1.
__device__ inline void store_row_chunk(uint16_t *Y, int64_t e0, const uint16_t *src, int count, int ci,
                                       int yshift) {
    const int64_t first = ((e0 + yshift) & ~int64_t(7)) - yshift;
    const int64_t c0 = first + 8 * (int64_t)ci;
    if (c0 >= e0 + count) return;
    uint16_t v[8];
    bool all = true;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int m = (int)(c0 + q - e0);
        const bool in = m >= 0 && m < count;
        v[q] = in ? src[m] : (uint16_t)0;
        all = all && in;
    }
    uint16_t *dst = Y + c0;
    if (all) {
        *reinterpret_cast<uint4 *>(dst) =
            make_uint4(v[0] | ((uint32_t)v[1] << 16), v[2] | ((uint32_t)v[3] << 16),
                       v[4] | ((uint32_t)v[5] << 16), v[6] | ((uint32_t)v[7] << 16));
        return;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int m = (int)(c0 + q - e0);
        if (m >= 0 && m < count) dst[q] = v[q];
    }
}

}  // namespace sa
