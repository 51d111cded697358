// Device helpers shared by the gfx950 kernels: wavefront / workgroup
// reductions and scans with a fixed combination order (so results are
// bitwise reproducible), exact division by a runtime constant, and bf16
// rounding.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace sa {

constexpr int kWave = 64;

// Sum over the 64 lanes of a wavefront with a fixed butterfly order; every
// lane receives the same value.
__device__ inline double wave_sum(double x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, kWave);
    return x;
}

__device__ inline uint32_t wave_sum_u32(uint32_t x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, kWave);
    return x;
}

// Minimum / maximum over the 64 lanes of a wavefront; every lane receives it.
__device__ inline int wave_min_i32(int x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x = min(x, __shfl_xor(x, off, kWave));
    return x;
}

__device__ inline int wave_max_i32(int x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x = max(x, __shfl_xor(x, off, kWave));
    return x;
}

// Inclusive prefix sum over the lanes of a wavefront (lane order).
__device__ inline uint32_t wave_incl_scan(uint32_t x) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        uint32_t y = __shfl_up(x, off, kWave);
        if (lane >= off) x += y;
    }
    return x;
}

// Exclusive prefix sum over the threads of a workgroup in thread order.
// `tmp` must hold blockDim.x / 64 + 1 words of LDS.  Returns the exclusive
// prefix; *total receives the workgroup total.  Contains barriers: every
// thread of the workgroup must call it.
__device__ inline uint32_t block_excl_scan(uint32_t x, uint32_t *tmp, uint32_t *total) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x >> 6;
    const int nwaves = blockDim.x >> 6;
    uint32_t incl = wave_incl_scan(x);
    if (lane == kWave - 1) tmp[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        uint32_t t = lane < nwaves ? tmp[lane] : 0u;
        uint32_t ti = wave_incl_scan(t);
        if (lane < nwaves) tmp[lane] = ti - t;  // exclusive per wave
        if (lane == nwaves - 1) tmp[nwaves] = ti;
    }
    __syncthreads();
    uint32_t r = tmp[wave] + incl - x;
    *total = tmp[nwaves];
    __syncthreads();
    return r;
}

// Exact floor(n / d) for 0 <= n < 2^31 and 1 <= d < 2^31 with a multiplier
// m = ceil(2^(31+l) / d), l = ceil(log2 d) (Granlund & Montgomery, "Division
// by invariant integers using multiplication", 1994, Theorem 4.2).
struct FastDiv {
    uint64_t mul;
    uint32_t shift;  // 31 + l
    uint32_t d;
};

inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while ((uint64_t(1) << l) < d) ++l;
    FastDiv f;
    f.shift = 31 + l;
    f.mul = ((uint64_t(1) << f.shift) + d - 1) / d;
    f.d = d;
    return f;
}

__device__ __host__ inline uint32_t fdiv(uint32_t n, const FastDiv &f) {
    return (uint32_t)(((uint64_t)n * f.mul) >> f.shift);
}

// binary32 -> bfloat16 bits, round to nearest even (the gfx950 convert).
__device__ inline uint16_t f32_to_bf16_bits(float x) {
    __bf16 h = (__bf16)x;
    return __builtin_bit_cast(uint16_t, h);
}

}  // namespace sa
