// gfx950 implicit-GEMM CONV over the compacted weight matrix (Section 3:
// after row / column pruning the CONV is still a full GEMM, only smaller).
//
// Per conv group g the GEMM is  Y^T[m, px] = sum_k Wc_g[m, k] * Xcol[px, k]
// with px = (n, p, q) an output pixel and k a kept (tap, channel) column.
//
// k_conv (the contraction, MFMA v_mfma_f32_32x32x16_bf16):
//   - A operand = Wc rows (kept filters), B operand = Xcol rows (output
//     pixels), fp32 accumulators; the two 64-wide K-slice tiles are staged
//     through LDS with two buffers: the loads of slice s+2 are issued while
//     slice s is multiplied, one barrier per slice; LDS rows are padded by
//     16 bytes so fragment reads spread over the banks;
//   - global reads are raw buffer loads: 32-bit offsets, and rows past the
//     end of the compacted matrix read as zero in hardware (no branches);
//     compacted rows are padded to 64 columns, so no K check on the A side;
//   - B rows are read as 16-byte vectors of 8 channels straight from the NHWC
//     input when the group's columns are every tap times one run of input
//     channels (dense, filter- or channel-pruned layers): Xcol is never
//     materialised;
//   - the output tile is staged through LDS and written as 16-byte rows;
//   - workgroup ids are remapped so that each XCD (8 per MI355X, each with
//     its own L2) walks a contiguous range of output tiles.
// k_im2col (filter-shape pruning: arbitrary (tap, channel) columns, or inputs
// with few channels): writes the compacted Xcol rows [N*P*Q][ldk] to scratch
// first, then k_conv runs on them as a 1x1 convolution.  Each workgroup copies
// the input footprint of 64 output pixels (the channels the group reads,
// zero-padded halo) into LDS and gathers every kept column from there through
// a per-column byte-offset table, one lane per output pixel (consecutive
// pixels fall in consecutive LDS banks); k_im2col_global gathers straight
// from global memory when the footprint does not fit in LDS.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>

#include "sa_device.h"
#include "sa_host.h"
#include "structadmm.h"

namespace sa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBK = 64;            // K slice per stage (= compacted row padding)
constexpr int kRow = kBK + 8;      // LDS row of a staged operand tile (bf16 elements)
constexpr int kLdsBytes = 160 * 1024;
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

// ---------------------------------------------------------------- k_conv
// One conv group of a launch (every group of a layer runs in one launch).
struct ConvGroup {
    const uint16_t *X;   // NHWC input, or the group's gathered Xcol rows
    const uint16_t *Wc;  // group base
    uint32_t x_bytes;
    int32_t Cx, M, K, ldk, run, run_base, o_off, mtiles, begin;
    FastDiv divRun;
};
struct ConvArgs {
    uint16_t *Y;
    int32_t H, W, D, stride, pad, P, Q, NPQ, Cy;
    int32_t ngroups, nblocks;
    FastDiv divPQ, divQ, divD;
    ConvGroup g[SA_MAX_CONV_GROUPS];
};

template <int BM, int BN, int WN, int WM>
struct ConvCfg {
    static constexpr int NT = 64 * WN * WM;
    static constexpr int WTM = BN / WM, WTN = BM / WN;  // wavefront tile (m, px)
    static constexpr int TM = WTM / 32, TN = WTN / 32;
    static constexpr int AR = (BN * 8 + NT - 1) / NT;  // A chunks (16 B) per thread per slice
    static constexpr int BR = (BM * 8 + NT - 1) / NT;  // B chunks per thread per slice
    static constexpr int stage_bytes = 2 * (2 * BN * kRow + 2 * BM * kRow);
    static constexpr int c_bytes = 2 * BM * (BN + 8);
    static constexpr int lds = stage_bytes > c_bytes ? stage_bytes : c_bytes;
    static_assert(TM >= 1 && TN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "tile shape");
};

template <int BM, int BN, int WN, int WM>
__global__ __launch_bounds__(64 * WN * WM) void k_conv(ConvArgs a) {
    using Cfg = ConvCfg<BM, BN, WN, WM>;
    constexpr int NT = Cfg::NT, WTM = Cfg::WTM, WTN = Cfg::WTN, TM = Cfg::TM, TN = Cfg::TN;
    constexpr int AR = Cfg::AR, BR = Cfg::BR;

    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t *sA = reinterpret_cast<uint16_t *>(smem);  // [2][BN][kRow]
    uint16_t *sB = sA + 2 * BN * kRow;                  // [2][BM][kRow]

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wn = wave % WN, wm = wave / WN;

    int bid = blockIdx.x;
    if ((a.nblocks & 7) == 0) bid = (bid & 7) * (a.nblocks >> 3) + (bid >> 3);
    int gi = 0;
    while (gi + 1 < a.ngroups && bid >= a.g[gi + 1].begin) ++gi;
    const ConvGroup &G = a.g[gi];
    const int lb = bid - G.begin;
    const int mt = lb % G.mtiles, nt = lb / G.mtiles;
    const int m0 = mt * BN, n0 = nt * BM;
    const int nst = G.ldk / kBK;
    const int kc = tid & 7, rb = tid >> 3;
    const int frow = lane & 31, fk = (lane >> 5) * 8;

    // A operand: rows past M read as zero through the buffer range
    const __amdgpu_buffer_rsrc_t wrs = rsrc(G.Wc, (uint32_t)G.M * (uint32_t)G.ldk * 2u);
    uint32_t aoff[AR];
#pragma unroll
    for (int i = 0; i < AR; ++i) aoff[i] = ((uint32_t)(m0 + rb + i * (NT / 8)) * (uint32_t)G.ldk + kc * 8) * 2u;

    // B operand: the output pixel of each chunk row this thread loads
    int xh0[BR], xw0[BR];
    uint32_t xrow[BR];  // byte offset of (n, 0, 0, run_base) in X
#pragma unroll
    for (int i = 0; i < BR; ++i) {
        const int pxr = n0 + rb + i * (NT / 8);
        const int px = min(pxr, a.NPQ - 1);
        const int nn = (int)fdiv((uint32_t)px, a.divPQ);
        const int rem = px - nn * a.P * a.Q;
        const int p = (int)fdiv((uint32_t)rem, a.divQ);
        const int q = rem - p * a.Q;
        // rows past the output read nothing: push their pixel off the image
        xh0[i] = pxr < a.NPQ ? p * a.stride - a.pad : -(1 << 28);
        xw0[i] = q * a.stride - a.pad;
        xrow[i] = ((uint32_t)nn * a.H * a.W * G.Cx + G.run_base) * 2u;
    }

    const __amdgpu_buffer_rsrc_t xrs = rsrc(G.X, G.x_bytes);
    constexpr bool kARagged = AR * (NT / 8) > BN;
    constexpr bool kBRagged = BR * (NT / 8) > BM;
    uint4 wreg[AR], xreg[BR];
    auto load_stage = [&](int s) {
#pragma unroll
        for (int i = 0; i < AR; ++i) wreg[i] = bload16(wrs, aoff[i] + (uint32_t)s * (kBK * 2));
        // k = tap * run + ch; the 8 columns of a chunk share the tap
        const int k = s * kBK + kc * 8;
        const int tap = (int)fdiv((uint32_t)k, G.divRun);
        const int ch = k - tap * G.run;
        const int c = (int)fdiv((uint32_t)tap, a.divD);
        const int d = tap - c * a.D;
        const uint32_t delta = ((uint32_t)(c * a.W + d) * G.Cx + ch) * 2u;
        const bool kin = k < G.K;
#pragma unroll
        for (int i = 0; i < BR; ++i) {
            const int h = xh0[i] + c, w = xw0[i] + d;
            const bool in = kin && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
            // an offset past the end of the buffer reads as zero
            const uint32_t off =
                in ? xrow[i] + ((uint32_t)(xh0[i] * a.W + xw0[i]) * G.Cx) * 2u + delta : kInvalidOffset;
            xreg[i] = bload16(xrs, off);
        }
    };
    auto store_stage = [&](int buf) {
        uint16_t *A = sA + buf * BN * kRow;
        uint16_t *B = sB + buf * BM * kRow;
#pragma unroll
        for (int i = 0; i < AR; ++i) {
            const int r = rb + i * (NT / 8);
            if (!kARagged || r < BN) *reinterpret_cast<uint4 *>(&A[r * kRow + kc * 8]) = wreg[i];
        }
#pragma unroll
        for (int i = 0; i < BR; ++i) {
            const int r = rb + i * (NT / 8);
            if (!kBRagged || r < BM) *reinterpret_cast<uint4 *>(&B[r * kRow + kc * 8]) = xreg[i];
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    load_stage(0);
    store_stage(0);
    if (nst > 1) load_stage(1);
    __syncthreads();

    for (int s = 0; s < nst; ++s) {
        if (s + 1 < nst) store_stage((s + 1) & 1);
        if (s + 2 < nst) load_stage(s + 2);
        const uint16_t *A = sA + (s & 1) * BN * kRow;
        const uint16_t *B = sB + (s & 1) * BM * kRow;
#pragma unroll
        for (int kk = 0; kk < kBK; kk += 16) {
            bf16x8 af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const bf16x8 *>(&A[(wm * WTM + i * 32 + frow) * kRow + kk + fk]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bfr[j] = *reinterpret_cast<const bf16x8 *>(&B[(wn * WTN + j * 32 + frow) * kRow + kk + fk]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }

    // epilogue: accumulator (i, j, r): m = i*32 + (r/4)*8 + (lane/32)*4 + r%4, px = j*32 + lane%32
    uint16_t *sC = reinterpret_cast<uint16_t *>(smem);  // [BM][BN + 8]
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int ml = wm * WTM + i * 32 + r4 * 8 + (lane >> 5) * 4;
                const int pl = wn * WTN + j * 32 + (lane & 31);
                const uint32_t lo = (uint32_t)f32_to_bf16_bits(acc[i][j][r4 * 4 + 0]) |
                                    ((uint32_t)f32_to_bf16_bits(acc[i][j][r4 * 4 + 1]) << 16);
                const uint32_t hi = (uint32_t)f32_to_bf16_bits(acc[i][j][r4 * 4 + 2]) |
                                    ((uint32_t)f32_to_bf16_bits(acc[i][j][r4 * 4 + 3]) << 16);
                *reinterpret_cast<uint2 *>(&sC[pl * (BN + 8) + ml]) = make_uint2(lo, hi);
            }
    __syncthreads();
    const bool vec_out = (a.Cy % 8 == 0) && ((G.o_off + m0) % 8 == 0) && ((uintptr_t)a.Y % 16 == 0);
    constexpr int CPR = BN / 8;  // 16-byte chunks per output row
    for (int c = tid; c < BM * CPR; c += NT) {
        const int pl = c / CPR, mc = c - pl * CPR;
        const int px = n0 + pl, m = m0 + mc * 8;
        if (px >= a.NPQ || m >= G.M) continue;
        uint16_t *dst = a.Y + (int64_t)px * a.Cy + G.o_off + m;
        const uint16_t *srcp = &sC[pl * (BN + 8) + mc * 8];
        if (vec_out && m + 8 <= G.M) {
            *reinterpret_cast<uint4 *>(dst) = *reinterpret_cast<const uint4 *>(srcp);
        } else {
            for (int e = 0; e < 8 && m + e < G.M; ++e) dst[e] = srcp[e];
        }
    }
}

// ---------------------------------------------------------------- k_im2col
struct GatherArgs {
    const uint16_t *X;
    const int32_t *col_ch;   // group base
    const int32_t *col_tap;  // group base
    uint16_t *Xcol;          // [NPQ][ldk]
    int32_t N, H, W, Cx, C, D, stride, pad, P, Q, NPQ, K, ldk;
    uint32_t x_bytes;
    int32_t ch_lo, pix_bytes, Wp, Hp, patch_bytes, nch, vec16;
    FastDiv divQ, divP, divHp, divWpN, divNch;
};

constexpr int kGatherPx = 64;  // output pixels per workgroup (one per lane)
constexpr int kGatherThreads = 256;

// Compacted im2col rows of 64 output pixels, gathered from an LDS copy of
// their input footprint.  Columns k in [K, ldk) are written as +0.
__global__ __launch_bounds__(kGatherThreads) void k_im2col(GatherArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint8_t *patch = smem;
    int32_t *tab = reinterpret_cast<int32_t *>(smem + a.patch_bytes);
    const int tid = threadIdx.x;
    const int n0 = blockIdx.x * kGatherPx;
    // input rows (padded coordinates, images stacked) used by this tile
    const int r0 = (int)fdiv((uint32_t)n0, a.divQ);
    const int r1 = (int)fdiv((uint32_t)(min(n0 + kGatherPx, a.NPQ) - 1), a.divQ);
    const int i0 = (int)fdiv((uint32_t)r0, a.divP), i1 = (int)fdiv((uint32_t)r1, a.divP);
    const int g0 = i0 * a.Hp + (r0 - i0 * a.P) * a.stride;
    const int g1 = i1 * a.Hp + (r1 - i1 * a.P) * a.stride + a.C;  // exclusive
    const int total = (g1 - g0) * a.Wp * a.nch;
    const __amdgpu_buffer_rsrc_t xrs = rsrc(a.X, a.x_bytes);
    // batches of 8 loads per thread in flight before their LDS stores
    constexpr int kFill = 8;
    for (int base = tid; base < total; base += kGatherThreads * kFill) {
        uint4 v[kFill];
        int dst[kFill];
#pragma unroll
        for (int u = 0; u < kFill; ++u) {
            const int idx = base + u * kGatherThreads;
            dst[u] = -1;
            v[u] = make_uint4(0, 0, 0, 0);
            if (idx >= total) continue;
            const int pr = (int)fdiv((uint32_t)idx, a.divWpN);
            const int rem = idx - pr * a.Wp * a.nch;
            const int wc = (int)fdiv((uint32_t)rem, a.divNch);
            const int ch = rem - wc * a.nch;
            const int gr = g0 + pr;
            const int img = (int)fdiv((uint32_t)gr, a.divHp);
            const int h = gr - img * a.Hp - a.pad, w = wc - a.pad;
            const bool in = img < a.N && h >= 0 && h < a.H && w >= 0 && w < a.W;
            const uint32_t src = (((uint32_t)(img * a.H + h) * a.W + w) * a.Cx + a.ch_lo) * 2u;
            if (a.vec16) {
                if (in) v[u] = bload16(xrs, src + ch * 16);
                dst[u] = (pr * a.Wp + wc) * a.pix_bytes + ch * 16;
            } else {
                if (in) v[u].x = a.X[src / 2 + ch];
                dst[u] = (pr * a.Wp + wc) * a.pix_bytes + ch * 2;
            }
        }
#pragma unroll
        for (int u = 0; u < kFill; ++u) {
            if (dst[u] < 0) continue;
            if (a.vec16) {
                uint32_t *d32 = reinterpret_cast<uint32_t *>(patch + dst[u]);
                d32[0] = v[u].x;
                d32[1] = v[u].y;
                d32[2] = v[u].z;
                d32[3] = v[u].w;
            } else {
                *reinterpret_cast<uint16_t *>(patch + dst[u]) = (uint16_t)v[u].x;
            }
        }
    }
#pragma unroll 4
    for (int k = tid; k < a.ldk; k += kGatherThreads) {
        int32_t off = -1;  // padding column
        if (k < a.K) {
            const int t = a.col_tap[k];
            const int cc = t / a.D, d = t - cc * a.D;
            off = (cc * a.Wp + d) * a.pix_bytes + (a.col_ch[k] - a.ch_lo) * 2;
        }
        tab[k] = off;
    }
    __syncthreads();

    // one lane per output pixel; the four wavefronts take 8-column chunks in turn
    const int lane = tid & 63, wave = tid >> 6;
    const int px = n0 + lane;
    if (px >= a.NPQ) return;
    int pbase;
    {
        const int r = (int)fdiv((uint32_t)px, a.divQ);
        const int img = (int)fdiv((uint32_t)r, a.divP);
        const int q = px - r * a.Q;
        const int gr = img * a.Hp + (r - img * a.P) * a.stride;
        pbase = ((gr - g0) * a.Wp + q * a.stride) * a.pix_bytes;
    }
    const uint8_t *p = patch + pbase;
    uint16_t *row = a.Xcol + (int64_t)px * a.ldk;
    const int nchunk = a.ldk / 8;
#pragma unroll 2
    for (int c = wave; c < nchunk; c += kGatherThreads / 64) {
        const int4 o0 = *reinterpret_cast<const int4 *>(tab + c * 8);
        const int4 o1 = *reinterpret_cast<const int4 *>(tab + c * 8 + 4);
        const int off[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
        uint32_t v[8];
        if (c * 8 + 8 <= a.K) {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = *reinterpret_cast<const uint16_t *>(p + off[e]);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = off[e] >= 0 ? *reinterpret_cast<const uint16_t *>(p + off[e]) : 0u;
        }
        *reinterpret_cast<uint4 *>(row + c * 8) =
            make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
    }
}

// The same rows gathered element by element from global memory: inputs with
// few channels (8 consecutive columns of a kernel row are then contiguous in
// NHWC, so the reads coalesce) or footprints too large for LDS.  Threads
// take (pixel, 8-column chunk) pairs, chunk fastest; the column table
// (kernel row, kernel column, input channel) is held in LDS.
__global__ __launch_bounds__(256) void k_im2col_global(GatherArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint32_t *tab = reinterpret_cast<uint32_t *>(smem);  // [ldk]
    for (int k = threadIdx.x; k < a.ldk; k += 256) {
        uint32_t ent = 0xffffffffu;  // padding column
        if (k < a.K) {
            const int t = a.col_tap[k];
            const int cc = t / a.D, d = t - cc * a.D;
            ent = ((uint32_t)cc << 24) | ((uint32_t)d << 16) | (uint32_t)a.col_ch[k];
        }
        tab[k] = ent;
    }
    __syncthreads();
    const int nchunk = a.ldk / 8;
    const int64_t total = (int64_t)a.NPQ * nchunk;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        const int px = (int)(i / nchunk), c = (int)(i - (int64_t)px * nchunk);
        const int r = (int)fdiv((uint32_t)px, a.divQ);
        const int img = (int)fdiv((uint32_t)r, a.divP);
        const int h0 = (r - img * a.P) * a.stride - a.pad, w0 = (px - r * a.Q) * a.stride - a.pad;
        const uint16_t *xi = a.X + (int64_t)img * a.H * a.W * a.Cx;
        const uint4 t0 = *reinterpret_cast<const uint4 *>(tab + c * 8);
        const uint4 t1 = *reinterpret_cast<const uint4 *>(tab + c * 8 + 4);
        const uint32_t ent[8] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w};
        uint32_t v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            v[e] = 0;
            const uint32_t en = ent[e];
            const int h = h0 + (int)(en >> 24), w = w0 + (int)((en >> 16) & 255u);
            const int ch = (int)(en & 0xffffu);
            if (en != 0xffffffffu && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W && ch < a.Cx)
                v[e] = xi[(h * a.W + w) * a.Cx + ch];
        }
        *reinterpret_cast<uint4 *>(a.Xcol + (int64_t)px * a.ldk + c * 8) =
            make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
    }
}

// ---------------------------------------------------------------- host side
template <int BM, int BN, int WN, int WM>
int launch_conv(ConvArgs a, hipStream_t stream) {
    using Cfg = ConvCfg<BM, BN, WN, WM>;
    // blocks of group i: [begin, begin + mtiles * ntiles), m-tiles fastest
    const int ntiles = (a.NPQ + BM - 1) / BM;
    int begin = 0;
    for (int i = 0; i < a.ngroups; ++i) {
        a.g[i].mtiles = (a.g[i].M + BN - 1) / BN;
        a.g[i].begin = begin;
        begin += a.g[i].mtiles * ntiles;
    }
    a.nblocks = begin;
    auto kern = k_conv<BM, BN, WN, WM>;
    if (int rc = check_hip(hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::lds),
                           "conv: set LDS size"))
        return rc;
    hipLaunchKernelGGL(kern, dim3(a.nblocks), dim3(Cfg::NT), Cfg::lds, stream, a);
    return check_hip(hipGetLastError(), "k_conv");
}

// One launch for every group of a; the tile shape follows the widest group.
int run_conv(ConvArgs a, hipStream_t stream) {
    if (a.ngroups == 0) return SA_OK;
    bool all256 = true;
    int maxM = 0;
    for (int i = 0; i < a.ngroups; ++i) {
        a.g[i].divRun = make_fastdiv((uint32_t)std::max(1, a.g[i].run));  // a group without columns has run 0
        all256 = all256 && a.g[i].M % 256 == 0;
        maxM = std::max(maxM, a.g[i].M);
    }
    a.divPQ = make_fastdiv((uint32_t)(a.P * a.Q));
    a.divQ = make_fastdiv((uint32_t)a.Q);
    a.divD = make_fastdiv((uint32_t)a.D);
    if (all256) return launch_conv<128, 256, 2, 2>(a, stream);
    if (maxM > 64) return launch_conv<128, 128, 2, 2>(a, stream);
    if (maxM > 32) return launch_conv<256, 64, 4, 1>(a, stream);
    return launch_conv<256, 32, 4, 1>(a, stream);
}

bool is_vec(const sa_compact_sizes &s, int g, int Cx) {
    return s.run[g] > 0 && s.run[g] % 8 == 0 && s.run_base[g] % 8 == 0 && Cx % 8 == 0;
}

// Footprint of the largest output tile of BM pixels: padded input rows.
int patch_rows(int NPQ, int P, int Q, int Hp, int stride, int C, int BM) {
    int best = 0;
    for (int n0 = 0; n0 < NPQ; n0 += BM) {
        const int r0 = n0 / Q, r1 = (std::min(n0 + BM, NPQ) - 1) / Q;
        const int g0 = (r0 / P) * Hp + (r0 % P) * stride;
        const int g1 = (r1 / P) * Hp + (r1 % P) * stride + C;
        best = std::max(best, g1 - g0);
    }
    return best;
}

int gather_group(GatherArgs g, int ch_span, hipStream_t stream) {
    g.Wp = g.W + 2 * g.pad;
    g.Hp = g.H + 2 * g.pad;
    g.divQ = make_fastdiv((uint32_t)g.Q);
    g.divP = make_fastdiv((uint32_t)g.P);
    g.vec16 = (g.Cx % 8 == 0) && (g.ch_lo % 8 == 0);
    int bytes;
    if (g.vec16) {
        g.nch = (ch_span + 7) / 8;
        bytes = g.nch * 16;
    } else {
        g.nch = ch_span;
        bytes = (ch_span * 2 + 3) / 4 * 4;
    }
    if ((bytes / 4) % 2 == 0) bytes += 4;  // odd number of dwords per pixel: consecutive pixels, consecutive banks
    g.pix_bytes = bytes;
    const int64_t patch = (int64_t)patch_rows(g.NPQ, g.P, g.Q, g.Hp, g.stride, g.C, kGatherPx) * g.Wp * bytes;
    const int64_t lds = (patch + 15) / 16 * 16 + (int64_t)g.ldk * 4;
    const int blocks = (g.NPQ + kGatherPx - 1) / kGatherPx;
    // the LDS patch pays off when each pixel carries a few cache lines of channels
    if (ch_span >= 16 && lds <= kLdsBytes) {
        g.patch_bytes = (int)((patch + 15) / 16 * 16);
        g.divHp = make_fastdiv((uint32_t)g.Hp);
        g.divWpN = make_fastdiv((uint32_t)(g.Wp * g.nch));
        g.divNch = make_fastdiv((uint32_t)g.nch);
        if (int rc = check_hip(hipFuncSetAttribute(reinterpret_cast<const void *>(k_im2col),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds),
                               "conv: set LDS size"))
            return rc;
        hipLaunchKernelGGL(k_im2col, dim3(blocks), dim3(kGatherThreads), (size_t)lds, stream, g);
        return check_hip(hipGetLastError(), "k_im2col");
    }
    const int64_t chunks = (int64_t)g.NPQ * (g.ldk / 8);
    const size_t tab = (size_t)g.ldk * 4;
    if (int rc = check_hip(hipFuncSetAttribute(reinterpret_cast<const void *>(k_im2col_global),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)tab),
                           "conv: set LDS size"))
        return rc;
    hipLaunchKernelGGL(k_im2col_global, dim3((unsigned)std::min<int64_t>(8192, (chunks + 255) / 256)), dim3(256), tab,
                       stream, g);
    return check_hip(hipGetLastError(), "k_im2col_global");
}

// Validates the descriptor (beyond validate_conv) and returns the scratch size.
int conv_plan(const sa_conv_desc &d, size_t *ws_need) {
    if (int rc = validate_conv(d)) return rc;
    const sa_compact_sizes &s = *d.sizes;
    const int64_t P = ((int64_t)d.H + 2 * d.pad - d.C) / d.stride + 1;
    const int64_t Q = ((int64_t)d.W + 2 * d.pad - d.D) / d.stride + 1;
    const int64_t NPQ = (int64_t)d.N * P * Q;
    if (d.Cx > 65535) return fail(SA_E_UNSUPPORTED, "conv: Cx > 65535");
    if ((int64_t)d.N * d.H * d.W * d.Cx * 2 >= (int64_t(1) << 31))
        return fail(SA_E_UNSUPPORTED, "conv: input of 2 GiB or more");
    size_t need = 0;
    for (int g = 0; g < s.groups; ++g) {
        if (s.ldk[g] != (s.K[g] + kBK - 1) / kBK * kBK || s.wc_offset[g] % 8 != 0)
            return fail(SA_E_ARG, "conv: sizes->ldk / wc_offset of group %d are not those of structadmm_compact", g);
        if (((int64_t)s.M[g] + 256) * s.ldk[g] * 2 >= (int64_t(1) << 31))
            return fail(SA_E_UNSUPPORTED, "conv: compacted matrix of group %d of 2 GiB or more", g);
        if (s.K[g] > 0 && (s.ch_lo[g] < 0 || s.ch_span[g] <= 0 || s.ch_lo[g] + s.ch_span[g] > d.Cx))
            return fail(SA_E_ARG, "conv: channel span of group %d outside the input's %d channels", g, d.Cx);
        if (s.M[g] > 0 && !is_vec(s, g, d.Cx)) {
            const int64_t bytes = NPQ * s.ldk[g] * 2;
            if (bytes >= (int64_t(1) << 31))
                return fail(SA_E_UNSUPPORTED, "conv: gathered rows of group %d need 2 GiB or more", g);
            need += ((size_t)bytes + 255) / 256 * 256;  // each gathered group has its own rows
        }
    }
    *ws_need = need;
    return SA_OK;
}

}  // namespace
}  // namespace sa

using namespace sa;

extern "C" size_t structadmm_conv_workspace(const sa_conv_desc *desc) {
    if (!desc) return 0;
    size_t need = 0;
    if (conv_plan(*desc, &need) != SA_OK) {
        clear_error();
        return 0;
    }
    return need;
}

extern "C" int structadmm_conv_fwd(const sa_conv_desc *desc, hipStream_t stream) {
    clear_error();
    if (!desc) return fail(SA_E_ARG, "conv: desc is required");
    const sa_conv_desc &d = *desc;
    size_t need = 0;
    if (int rc = conv_plan(d, &need)) return rc;
    if (need > 0) {
        if (!d.ws || d.ws_bytes < need)
            return fail(SA_E_WORKSPACE, "conv: scratch of %zu bytes required (%zu given)", need, d.ws ? d.ws_bytes : 0);
        if (!aligned(d.ws, 256)) return fail(SA_E_ALIGN, "conv: scratch must be 256-byte aligned");
    }
    const sa_compact_sizes &s = *d.sizes;
    const int P = (d.H + 2 * d.pad - d.C) / d.stride + 1;
    const int Q = (d.W + 2 * d.pad - d.D) / d.stride + 1;
    const int NPQ = d.N * P * Q;
    const uint32_t x_bytes = (uint32_t)((int64_t)d.N * d.H * d.W * d.Cx * 2);
    int Cy = 0;
    for (int g = 0; g < s.groups; ++g) Cy += s.M[g];

    // groups read straight from the NHWC input share one launch; groups with
    // arbitrary columns are gathered first and share a second, 1x1 launch
    ConvArgs direct, gathered;
    memset(&direct, 0, sizeof direct);
    memset(&gathered, 0, sizeof gathered);
    direct.Y = gathered.Y = d.Y;
    direct.Cy = gathered.Cy = Cy;
    direct.NPQ = gathered.NPQ = NPQ;
    direct.H = d.H;
    direct.W = d.W;
    direct.D = d.D;
    direct.stride = d.stride;
    direct.pad = d.pad;
    direct.P = P;
    direct.Q = Q;
    gathered.H = gathered.W = gathered.D = gathered.stride = gathered.P = gathered.Q = 1;
    gathered.pad = 0;
    size_t ws_off = 0;
    for (int g = 0; g < s.groups; ++g) {
        if (s.M[g] == 0) continue;  // no output channels in this group
        const bool vec = is_vec(s, g, d.Cx);
        ConvArgs &a = vec ? direct : gathered;
        ConvGroup &G = a.g[a.ngroups++];
        G.Wc = d.Wc + s.wc_offset[g];
        G.M = s.M[g];
        G.ldk = s.ldk[g];
        G.o_off = s.row_offset[g];
        if (vec) {
            G.X = d.X;
            G.x_bytes = x_bytes;
            G.Cx = d.Cx;
            G.K = s.K[g];
            G.run = s.run[g];
            G.run_base = s.run_base[g];
            continue;
        }
        // the compacted im2col rows [N*P*Q][ldk] of this group, in its scratch region
        uint16_t *xcol = reinterpret_cast<uint16_t *>(static_cast<uint8_t *>(d.ws) + ws_off);
        const size_t bytes = (size_t)NPQ * s.ldk[g] * 2;
        ws_off += (bytes + 255) / 256 * 256;
        if (s.ldk[g] > 0) {  // a group without columns gathers nothing: its outputs are zero
            GatherArgs gth;
            memset(&gth, 0, sizeof gth);
            gth.X = d.X;
            gth.col_ch = d.col_ch + s.col_offset[g];
            gth.col_tap = d.col_tap + s.col_offset[g];
            gth.Xcol = xcol;
            gth.N = d.N;
            gth.H = d.H;
            gth.W = d.W;
            gth.Cx = d.Cx;
            gth.C = d.C;
            gth.D = d.D;
            gth.stride = d.stride;
            gth.pad = d.pad;
            gth.P = P;
            gth.Q = Q;
            gth.NPQ = NPQ;
            gth.K = s.K[g];
            gth.ldk = s.ldk[g];
            gth.x_bytes = x_bytes;
            gth.ch_lo = s.K[g] > 0 ? s.ch_lo[g] : 0;
            if (int rc = gather_group(gth, std::max(1, s.ch_span[g]), stream)) return rc;
        }
        G.X = xcol;
        G.x_bytes = (uint32_t)bytes;
        G.Cx = s.ldk[g];
        G.K = s.ldk[g];
        G.run = s.ldk[g];
        G.run_base = 0;
    }
    if (int rc = run_conv(direct, stream)) return rc;
    return run_conv(gathered, stream);
}
