// gfx950 implicit-GEMM CONV over the compacted weight matrix (Section 3:
// after row / column pruning the CONV is still a full GEMM, only smaller).
//
// Per conv group g the GEMM is  Y^T[m, px] = sum_k Wc_g[m, k] * Xcol[px, k]
// with px = (n, p, q) an output pixel and k a kept (tap, channel) column.
// structadmm_conv_fwd takes one of three paths per group, all on MFMA
// v_mfma_f32_32x32x16_bf16 (A = Wc rows, B = output pixels, fp32 accumulate;
// small ragged filter groups over a few hundred columns take the 16-row
// variant of the direct path in conv_ig.hip):
//
// k_conv (direct): the group's columns are every tap times one run of 8k
//   input channels (dense, filter- or channel-pruned layers); 128-pixel tiles
//   of 128 or 64 filters with eight wavefronts.  B rows are read
//   as 16-byte vectors straight from the NHWC input; both operand tiles are
//   staged through LDS in two buffers of 64 columns (loads of slice s+2 in
//   flight while slice s is multiplied); raw buffer loads with 32-bit offsets
//   read rows past the matrix as zero, without branches.
// k_conv_patch (fused gather): arbitrary (tap, channel) columns over inputs
//   whose channels are 8-aligned (filter-shape pruning).  Each workgroup copies
//   the input footprint of its pixels into LDS once and its wavefronts gather
//   their B fragments from that copy through a per-column offset table.
// k_im2col / k_im2col_global + k_conv (two-phase): inputs with few channels
//   or footprints too large for LDS; the compacted im2col rows [N*P*Q][ldk]
//   go to caller scratch first, then k_conv runs on them as a 1x1 convolution.
//   k_im2col gathers from an LDS copy of the footprint of 64 output pixels,
//   k_im2col_global straight from global memory.
// Every path launches once per layer for all of its conv groups, stages the
// output tile through LDS for 16-byte stores, and remaps workgroup ids so that
// each XCD (8 per MI355X, each with its own L2) walks a contiguous range of
// tiles.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <set>
#include <tuple>
#include <utility>

#include "conv_ig.h"
#include "sa_conv_device.h"
#include "sa_device.h"
#include "sa_host.h"
#include "structadmm.h"

namespace sa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int kBK = 64;            // K slice per stage (= compacted row padding)
constexpr int kRow = kBK + 8;      // LDS row of a staged operand tile (bf16 elements)
constexpr int kLdsBytes = 160 * 1024;

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
    float *part;          // split K: binary32 partial sums [ksplit][part_stride]
    int64_t part_stride;  // floats per chunk (N*P*Q*Cy rounded up to 4)
    int32_t ksplit, base_blocks;
    int32_t H, W, D, stride, pad, P, Q, NPQ, Cy;
    int32_t ldy;  // Y's row pitch (>= Cy)
    int32_t ngroups, nblocks;
    FastDiv divPQ, divQ, divD, divCy;
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

template <int BM, int BN, int WN, int WM, bool SPLIT>
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
    bid = xcd_remap(bid, a.nblocks);
    int chunk = 0;  // split K: the chunk of column slices this workgroup sums
    if constexpr (SPLIT) {
        chunk = bid / a.base_blocks;
        bid -= chunk * a.base_blocks;
    }
    int gi = 0;
    while (gi + 1 < a.ngroups && bid >= a.g[gi + 1].begin) ++gi;
    const ConvGroup &G = a.g[gi];
    const int lb = bid - G.begin;
    const int mt = lb % G.mtiles, nt = lb / G.mtiles;
    const int m0 = mt * BN, n0 = nt * BM;
    int s_begin = 0, s_end = G.ldk / kBK;
    if constexpr (SPLIT) {
        const int nst = s_end;
        s_begin = nst * chunk / a.ksplit;
        s_end = nst * (chunk + 1) / a.ksplit;
    }
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

    load_stage(s_begin);
    store_stage(0);
    if (s_begin + 1 < s_end) load_stage(s_begin + 1);
    __syncthreads();

    for (int s = s_begin; s < s_end; ++s) {
        if (s + 1 < s_end) store_stage((s + 1 - s_begin) & 1);
        if (s + 2 < s_end) load_stage(s + 2);
        const uint16_t *A = sA + ((s - s_begin) & 1) * BN * kRow;
        const uint16_t *B = sB + ((s - s_begin) & 1) * BM * kRow;
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
    if constexpr (SPLIT) {  // binary32 partial sums of this chunk; k_splitk_sum adds the chunks
        float *part = a.part + (int64_t)chunk * a.part_stride;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    const int m = m0 + wm * WTM + i * 32 + r4 * 8 + (lane >> 5) * 4;
                    const int px = n0 + wn * WTN + j * 32 + (lane & 31);
                    if (px >= a.NPQ) continue;
                    float *dst = part + (int64_t)px * a.Cy + G.o_off + m;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (m + e < G.M) dst[e] = acc[i][j][r4 * 4 + e];
                }
        return;
    }
    uint16_t *sC = reinterpret_cast<uint16_t *>(smem);  // [BM][BN + 8]
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int ml = wm * WTM + i * 32 + r4 * 8 + (lane >> 5) * 4;
                const int pl = wn * WTN + j * 32 + (lane & 31);
                bf16x4 o;
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = (__bf16)acc[i][j][r4 * 4 + e];  // round to nearest even
                *reinterpret_cast<bf16x4 *>(&sC[pl * (BN + 8) + ml]) = o;
            }
    __syncthreads();
    if (a.Cy % 8 != 0 && a.ldy == a.Cy && G.mtiles == 1 && G.M == a.Cy && ((uintptr_t)a.Y & 15) == 0) {
        // whole, unaligned rows
        store_tile_rows<BN + 8>(a.Y, sC, n0, min(BM, a.NPQ - n0), a.Cy, a.divCy, tid, NT);
        return;
    }
    // the last channels of a row may run on into the row's padding (staged
    // rows past the group's filters hold +0)
    const int lim = G.o_off + G.M == a.Cy ? a.ldy - G.o_off : G.M;
    constexpr int CPR = BN / 8;  // 16-byte chunks per output row
    for (int c = tid; c < BM * CPR; c += NT) {
        const int pl = c / CPR, mc = c - pl * CPR;
        const int px = n0 + pl, m = m0 + mc * 8;
        if (px >= a.NPQ || m >= G.M) continue;
        uint16_t *dst = a.Y + (int64_t)px * a.ldy + G.o_off + m;
        store_out8(dst, &sC[pl * (BN + 8) + mc * 8], min(8, lim - m));
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

// ---------------------------------------------------------------- k_conv_patch
// Gathered groups without a scratch pass.  A workgroup owns the output tile
// (32*TM filters) x (32*NW*TN pixels) of one conv group, NW wavefronts (4, or
// 6 when that saves a round of workgroups over the CUs):
//   1. the input footprint of its pixels (the group's channel span, zero
//      halo) is copied once into LDS; for stride s > 1 the padded columns are
//      stored de-interleaved (column w at (w mod s) * Ws + w div s), so the
//      pixels of an output row read consecutive LDS words at every tap;
//   2. a per-column table holds the byte offset of (tap, channel) relative to
//      a pixel's base in that copy;
//   3. each wavefront owns 32*TN pixels and gathers its MFMA B fragments
//      straight from the copy into registers (lane = pixel, 8 columns per
//      lane), while the weight slices (A) are staged through LDS, two
//      buffers of 32 columns, shared by the wavefronts.
// Only ceil(K/16) column steps are run; columns past K in the last step are
// zeroed in registers, so padding never multiplies a value from the input.
constexpr int kPatchSlice = 32;                // columns per staged weight slice
constexpr int kPatchRowA = kPatchSlice + 8;    // LDS row of a weight slice (80 B)

struct PatchGroup {
    const uint16_t *Wc;      // group base, rows of ldk columns
    const int32_t *col_ch;   // group base
    const int32_t *col_tap;  // group base
    int32_t M, K, ldk, o_off, ch_lo, nch, pix_bytes, mtiles, begin;
    FastDiv divNch;          // 16-byte chunks per pixel
};
struct PatchArgs {
    const uint16_t *X;
    uint16_t *Y;
    uint32_t x_bytes;
    int32_t N, H, W, Cx, C, D, stride, pad, P, Q, NPQ, Cy;
    int32_t ldy;  // Y's row pitch (>= Cy)
    int32_t Hp, Wp, Ws, Wpp;
    int32_t ngroups, nblocks, patch_bytes, tab_bytes;
    // space-to-depth input (s2d > 1): X holds s x s blocks of the padded input
    // as s*s*Cxo channels; column (kh, kw, c) of the compacted matrix reads
    // tap (kh / s, kw / s), channel ((kh % s) * s + kw % s) * Cxo + c
    int32_t s2d, Do, Cxo;
    FastDiv divQ, divP, divHp, divD, divS, divDo, divS2d, divCy;
    PatchGroup g[SA_MAX_CONV_GROUPS];
};

template <int TM, int TN, int NW>
struct PatchCfg {
    static constexpr int NT = 64 * NW;         // NW wavefronts
    static constexpr int BNB = 32 * TM;        // filters per tile
    static constexpr int BMB = 32 * NW * TN;   // pixels per tile
    static constexpr int AR = (BNB * (kPatchSlice / 8) + NT - 1) / NT;  // 16-B weight chunks per thread
    static constexpr int a_bytes = 2 * BNB * kPatchRowA * 2;
    static constexpr int c_bytes = BMB * (BNB + 8) * 2;
};

template <int TM, int TN, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(TM >= 6 && NW <= 4 ? 1 : 2))) void k_conv_patch(PatchArgs a) {
    using Cfg = PatchCfg<TM, TN, NW>;
    constexpr int NT = Cfg::NT, BNB = Cfg::BNB, BMB = Cfg::BMB, AR = Cfg::AR;
    constexpr int CPS = kPatchSlice / 8;  // 16-B chunks per weight row of a slice

    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint8_t *patch = smem;
    int32_t *tab = reinterpret_cast<int32_t *>(smem + a.patch_bytes);
    uint16_t *sA = reinterpret_cast<uint16_t *>(smem + a.patch_bytes + a.tab_bytes);  // [2][BNB][kPatchRowA]

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;

    int bid = blockIdx.x;
    bid = xcd_remap(bid, a.nblocks);
    int gi = 0;
    while (gi + 1 < a.ngroups && bid >= a.g[gi + 1].begin) ++gi;
    const PatchGroup &G = a.g[gi];
    const int lb = bid - G.begin;
    const int mt = lb % G.mtiles, nt = lb / G.mtiles;
    const int m0 = mt * BNB, n0 = nt * BMB;

    // weight slices: issued first, they do not depend on the copy
    const __amdgpu_buffer_rsrc_t wrs = rsrc(G.Wc, (uint32_t)G.M * (uint32_t)G.ldk * 2u);
    uint32_t aoff[AR];
#pragma unroll
    for (int i = 0; i < AR; ++i) {
        const int c = tid + i * NT;
        aoff[i] = ((uint32_t)(m0 + c / CPS) * (uint32_t)G.ldk + (c % CPS) * 8) * 2u;
    }
    uint4 wreg[AR];
    auto load_a = [&](int s) {
#pragma unroll
        for (int i = 0; i < AR; ++i) wreg[i] = bload16(wrs, aoff[i] + (uint32_t)s * (kPatchSlice * 2));
    };
    auto store_a = [&](int buf) {
        uint16_t *A = sA + buf * BNB * kPatchRowA;
#pragma unroll
        for (int i = 0; i < AR; ++i) {
            const int c = tid + i * NT;
            if (BNB * CPS % NT == 0 || c < BNB * CPS)
                *reinterpret_cast<uint4 *>(&A[(c / CPS) * kPatchRowA + (c % CPS) * 8]) = wreg[i];
        }
    };
    // 32-column slices of two MFMA steps; the table covers two slices more,
    // so the offsets and B fragments ahead of the last step are read unconditionally
    const int nsl = (G.K + kPatchSlice - 1) / kPatchSlice;
    load_a(0);

    // 1. input footprint: padded rows [g0, g1) of the stacked padded images
    const int r0 = (int)fdiv((uint32_t)n0, a.divQ);
    const int r1 = (int)fdiv((uint32_t)(min(n0 + BMB, a.NPQ) - 1), a.divQ);
    const int i0 = (int)fdiv((uint32_t)r0, a.divP), i1 = (int)fdiv((uint32_t)r1, a.divP);
    const int g0 = i0 * a.Hp + (r0 - i0 * a.P) * a.stride;
    const int g1 = i1 * a.Hp + (r1 - i1 * a.P) * a.stride + a.C;  // exclusive
    const int nch = G.nch, pixb = G.pix_bytes;
    const __amdgpu_buffer_rsrc_t xrs = rsrc(a.X, a.x_bytes);

    // 2. column table: (kernel row, kernel column, channel) -> byte offset.
    // Its sources are read before the copy's loads are issued, so both wait
    // on one memory round trip.
    const int ntab = (nsl + 2) * kPatchSlice;
    auto tab_entry = [&](int k, int t, int ch) {
        int c, d;
        if (a.s2d > 1) {
            const int kh = (int)fdiv((uint32_t)t, a.divDo), kw = t - kh * a.Do;
            c = (int)fdiv((uint32_t)kh, a.divS2d);
            d = (int)fdiv((uint32_t)kw, a.divS2d);
            ch += ((kh - c * a.s2d) * a.s2d + (kw - d * a.s2d)) * a.Cxo;
        } else {
            c = (int)fdiv((uint32_t)t, a.divD);
            d = t - c * a.D;
        }
        const int dph = (int)fdiv((uint32_t)d, a.divS);
        tab[k] = (c * a.Wpp + (d - dph * a.stride) * a.Ws + dph) * pixb + (ch - G.ch_lo) * 2;
    };
    constexpr int kTabRegs = 4;  // entries per thread held across the copy's loads
    int ttap[kTabRegs], tch[kTabRegs];
#pragma unroll
    for (int q = 0; q < kTabRegs; ++q) {
        const int k = tid + q * NT;
        ttap[q] = 0;
        tch[q] = 0;
        if (k < G.K) {
            ttap[q] = G.col_tap[k];
            tch[q] = G.col_ch[k];
        }
    }

    // 1. the copy.  Every padded row is split the same way over the threads:
    //    item e of a row is chunk c of padded column 4*b + (e mod 4), with
    //    (b, c) = divmod(e / 4, nch), so the 64 lanes of a wavefront hold 16
    //    consecutive chunks of 4 neighbouring columns (256-byte runs of the
    //    input); with an odd number of words per pixel, the 4-byte LDS writes
    //    of a half-wavefront fall on distinct banks for most channel counts at
    //    stride 1, and on at most two lanes per bank otherwise (checked on the
    //    host for 1..64 chunks per pixel).  A thread's items of a row (two per
    //    pass) keep their source and LDS offsets across rows; the row's own
    //    terms (image, input row, zero halo) are the same for every thread.
    const int nrows = g1 - g0;
    const int rowitems = 4 * nch * ((a.Wp + 3) >> 2);
    const int J = (rowitems + NT - 1) / NT;  // items of a row per thread
    const int rowb = a.Wpp * pixb;           // LDS bytes per padded row
    const uint32_t rowsrc = (uint32_t)a.W * (uint32_t)a.Cx * 2u;
    constexpr int kRows = 16;  // rows per batch: up to 2 * kRows 16-byte loads in flight per thread
    for (int j0 = 0; j0 < J; j0 += 2) {
        const bool two = j0 + 1 < J;
        uint32_t so[2];  // source offset within the input row; past the buffer for the zero halo
        int cpo[2];      // LDS offset within the padded row; -1: no item
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
            const int e = tid + (j0 + jj) * NT;
            so[jj] = kInvalidOffset;
            cpo[jj] = -1;
            if (j0 + jj < J && e < rowitems) {
                const int q = e >> 2;
                const int b = (int)fdiv((uint32_t)q, G.divNch);
                const int c = q - b * nch;
                const int wpad = 4 * b + (e & 3);
                if (wpad < a.Wp) {
                    const int jw = (int)fdiv((uint32_t)wpad, a.divS);
                    cpo[jj] = ((wpad - jw * a.stride) * a.Ws + jw) * pixb + c * 16;
                    const int w = wpad - a.pad;
                    if ((unsigned)w < (unsigned)a.W) so[jj] = ((uint32_t)w * (uint32_t)a.Cx + G.ch_lo + c * 8) * 2u;
                }
            }
        }
        for (int pr0 = 0; pr0 < nrows; pr0 += kRows) {
            uint4 v[kRows][2];
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const int pr = pr0 + r;
                const int gr = g0 + pr;
                const int img = (int)fdiv((uint32_t)gr, a.divHp);
                const int h = gr - img * a.Hp - a.pad;
                const bool in = pr < nrows && img < a.N && (unsigned)h < (unsigned)a.H;
                const uint32_t sb = (uint32_t)(img * a.H + h) * rowsrc;  // below 2^31 when in
#pragma unroll
                for (int jj = 0; jj < 2; ++jj) {
                    v[r][jj] = make_uint4(0, 0, 0, 0);
                    if (in && (jj == 0 || two)) v[r][jj] = bload16(xrs, sb + so[jj]);
                }
            }
            if (j0 == 0 && pr0 == 0) {  // while the first loads are in flight: the table
#pragma unroll
                for (int q = 0; q < kTabRegs; ++q) {
                    const int k = tid + q * NT;
                    if (k < ntab) {
                        if (k < G.K) tab_entry(k, ttap[q], tch[q]);
                        else tab[k] = 0;  // columns past K: zeroed after the gather
                    }
                }
            }
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const int pr = pr0 + r;
                if (pr >= nrows) continue;
#pragma unroll
                for (int jj = 0; jj < 2; ++jj) {
                    if (cpo[jj] < 0) continue;
                    uint32_t *d32 = reinterpret_cast<uint32_t *>(patch + pr * rowb + cpo[jj]);
                    d32[0] = v[r][jj].x;
                    d32[1] = v[r][jj].y;
                    d32[2] = v[r][jj].z;
                    d32[3] = v[r][jj].w;
                }
            }
        }
    }
    for (int k = tid + kTabRegs * NT; k < ntab; k += NT) {  // long rows: the rest of the table
        if (k < G.K) tab_entry(k, G.col_tap[k], G.col_ch[k]);
        else tab[k] = 0;
    }
    store_a(0);
    if (nsl > 1) load_a(1);

    // byte offset of each owned pixel's window corner in the copy
    int pbase[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int px = n0 + wave * 32 * TN + j * 32 + (lane & 31);
        pbase[j] = 0;  // pixels past the output read the copy's first word; never stored
        if (px < a.NPQ) {
            const int r = (int)fdiv((uint32_t)px, a.divQ);
            const int img = (int)fdiv((uint32_t)r, a.divP);
            const int gr = img * a.Hp + (r - img * a.P) * a.stride;
            pbase[j] = ((gr - g0) * a.Wpp + (px - r * a.Q)) * pixb;
        }
    }
    __syncthreads();

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int frow = lane & 31, fk = (lane >> 5) * 8;
    // B fragments of the 16 columns from k0: lane = pixel, 8 columns per lane;
    // the column offsets are read one step before the gather that uses them
    struct Offs {
        int4 lo, hi;
    };
    auto offsets = [&](int k0) {
        Offs o;
        o.lo = *reinterpret_cast<const int4 *>(tab + k0 + fk);
        o.hi = *reinterpret_cast<const int4 *>(tab + k0 + fk + 4);
        return o;
    };
    auto gather = [&](int k0, const Offs &o, bf16x8 (&b)[TN]) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const uint8_t *pp = patch + pbase[j];
            u16x8 v;
            v[0] = *reinterpret_cast<const uint16_t *>(pp + o.lo.x);
            v[1] = *reinterpret_cast<const uint16_t *>(pp + o.lo.y);
            v[2] = *reinterpret_cast<const uint16_t *>(pp + o.lo.z);
            v[3] = *reinterpret_cast<const uint16_t *>(pp + o.lo.w);
            v[4] = *reinterpret_cast<const uint16_t *>(pp + o.hi.x);
            v[5] = *reinterpret_cast<const uint16_t *>(pp + o.hi.y);
            v[6] = *reinterpret_cast<const uint16_t *>(pp + o.hi.z);
            v[7] = *reinterpret_cast<const uint16_t *>(pp + o.hi.w);
            if (k0 + 16 > G.K) {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (k0 + fk + e >= G.K) v[e] = 0;
            }
            b[j] = __builtin_bit_cast(bf16x8, v);
        }
    };
    auto mma = [&](const bf16x8 (&af)[TM], const bf16x8 (&b)[TN]) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], b[j], acc[i][j], 0, 0, 0);
    };
    auto afrag = [&](const uint16_t *A, int kk, bf16x8 (&af)[TM]) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
            af[i] = *reinterpret_cast<const bf16x8 *>(&A[(i * 32 + frow) * kPatchRowA + kk + fk]);
    };
    // software pipeline over 16-column steps t: the weight fragments of t are
    // read first, then the offsets of t+2 and the gather of t+1 are issued,
    // and the MFMAs of t run while those reads are in flight
    bf16x8 b0[TN], b1[TN], af[TM];
    Offs o1 = offsets(0);
    gather(0, o1, b0);
    o1 = offsets(16);
    for (int s = 0; s < nsl; ++s) {
        if (s + 1 < nsl) store_a((s + 1) & 1);
        if (s + 2 < nsl) load_a(s + 2);
        const uint16_t *A = sA + (s & 1) * BNB * kPatchRowA;
        const int k0 = s * kPatchSlice;
        afrag(A, 0, af);
        Offs o2 = offsets(k0 + 32);
        gather(k0 + 16, o1, b1);
        mma(af, b0);
        afrag(A, 16, af);
        o1 = offsets(k0 + 48);
        gather(k0 + 32, o2, b0);
        mma(af, b1);
        __syncthreads();
    }

    // epilogue: accumulator (i, j, r): m = i*32 + (r/4)*8 + (lane/32)*4 + r%4,
    // px = wave*32*TN + j*32 + lane%32; staged through LDS as [px][m]
    uint16_t *sC = reinterpret_cast<uint16_t *>(smem);  // [BMB][BNB + 8]
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int ml = i * 32 + r4 * 8 + (lane >> 5) * 4;
                const int pl = wave * 32 * TN + j * 32 + (lane & 31);
                bf16x4 o;
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = (__bf16)acc[i][j][r4 * 4 + e];  // round to nearest even
                *reinterpret_cast<bf16x4 *>(&sC[pl * (BNB + 8) + ml]) = o;
            }
    __syncthreads();
    if (a.Cy % 8 != 0 && a.ldy == a.Cy && G.mtiles == 1 && G.M == a.Cy && ((uintptr_t)a.Y & 15) == 0) {
        // whole, unaligned rows
        store_tile_rows<BNB + 8>(a.Y, sC, n0, min(BMB, a.NPQ - n0), a.Cy, a.divCy, tid, NT);
        return;
    }
    // the last channels of a row may run on into the row's padding (+0)
    const int lim = G.o_off + G.M == a.Cy ? a.ldy - G.o_off : G.M;
    constexpr int CPR = BNB / 8;
    for (int c = tid; c < BMB * CPR; c += NT) {
        const int pl = c / CPR, mc = c - pl * CPR;
        const int px = n0 + pl, m = m0 + mc * 8;
        if (px >= a.NPQ || m >= G.M) continue;
        uint16_t *dst = a.Y + (int64_t)px * a.ldy + G.o_off + m;
        store_out8(dst, &sC[pl * (BNB + 8) + mc * 8], min(8, lim - m));
    }
}

// ---------------------------------------------------------------- k_splitk_sum
// Split K: Y = bf16(sum over chunks c = 0, 1, ... of part[c]) in that order
// (one fixed order: the result does not depend on which chunk finished
// first).  Element f = r * Cy + c of a chunk is output (row r, channel c),
// at Y[r * ldy + c].
__global__ __launch_bounds__(256) void k_splitk_sum(const float *part, int64_t stride, int ksplit, uint16_t *Y,
                                                     int64_t total, int Cy, int ldy) {
    const int64_t f = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (f >= total) return;
    if (ldy != Cy) {  // padded rows: element by element
        for (int64_t e = f; e < f + 4 && e < total; ++e) {
            float acc = part[e];
            for (int c = 1; c < ksplit; ++c) acc += part[c * stride + e];
            const int64_t r = e / Cy;
            Y[r * ldy + (e - r * Cy)] = f32_to_bf16_bits(acc);
        }
        return;
    }
    if (f + 4 <= total) {
        float4 acc = *reinterpret_cast<const float4 *>(part + f);
#pragma unroll 7
        for (int c = 1; c < ksplit; ++c) {
            const float4 v = *reinterpret_cast<const float4 *>(part + c * stride + f);
            acc.x += v.x;
            acc.y += v.y;
            acc.z += v.z;
            acc.w += v.w;
        }
        uint32_t *dst = reinterpret_cast<uint32_t *>(Y + f);  // Y is 4-byte aligned, f a multiple of 4
        dst[0] = (uint32_t)f32_to_bf16_bits(acc.x) | ((uint32_t)f32_to_bf16_bits(acc.y) << 16);
        dst[1] = (uint32_t)f32_to_bf16_bits(acc.z) | ((uint32_t)f32_to_bf16_bits(acc.w) << 16);
        return;
    }
    for (int64_t e = f; e < total; ++e) {
        float acc = part[e];
        for (int c = 1; c < ksplit; ++c) acc += part[c * stride + e];
        Y[e] = f32_to_bf16_bits(acc);
    }
}

// ---------------------------------------------------------------- k_s2d
// Space-to-depth image of the zero-padded input for layers with few channels:
// Xs[n][i][j][(a*s + b)*Cx + c] = Xpad[n][i*s + a][j*s + b][c], channels from
// s*s*Cx up to the next multiple of 8 zero.  The CONV over X (stride s) is then
// a stride-1 CONV over Xs with ceil(C/s) x ceil(D/s) taps, which k_conv_patch
// runs; s = 1 only pads the channels (and folds the zero border in).
struct S2dArgs {
    const uint16_t *X;
    uint16_t *Xs;
    int32_t N, H, W, Cx, s, pad, Hs, Ws, Cs, Creal;  // Creal = s*s*Cx, Cs = Creal rounded up to 8
    int32_t chunks;                           // N*Hs*Ws*Cs / 8 (< 2^27: the image is below 2 GiB)
    uint32_t x_bytes;                         // bytes of X (below 2 GiB)
    int32_t runs;                             // k_s2d_rows: copy whole runs (see there)
    FastDiv divCs8, divWs, divHs, divCx, divS;
};

// One thread per 8 consecutive channels (16 bytes) of the output image.
__global__ __launch_bounds__(256) void k_s2d(S2dArgs a) {
    const int cs8 = a.Cs / 8;
    for (int e = blockIdx.x * 256 + threadIdx.x; e < a.chunks; e += gridDim.x * 256) {
        const int pix = (int)fdiv((uint32_t)e, a.divCs8);  // (n, i, j)
        const int c0 = (e - pix * cs8) * 8;
        const int ni = (int)fdiv((uint32_t)pix, a.divWs);
        const int j = pix - ni * a.Ws;
        const int n = (int)fdiv((uint32_t)ni, a.divHs);
        const int i = ni - n * a.Hs;
        // channel c0 = (ra * s + rb) * Cx + c, advanced one channel at a time
        int blk = (int)fdiv((uint32_t)c0, a.divCx);
        int c = c0 - blk * a.Cx;
        int ra = (int)fdiv((uint32_t)blk, a.divS);
        int rb = blk - ra * a.s;
        const int64_t img = (int64_t)n * a.H * a.W;
        uint32_t v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int h = i * a.s + ra - a.pad, w = j * a.s + rb - a.pad;
            v[q] = (c0 + q < a.Creal && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W)
                       ? a.X[(img + (int64_t)h * a.W + w) * a.Cx + c]
                       : 0u;
            if (++c == a.Cx) {
                c = 0;
                if (++rb == a.s) {
                    rb = 0;
                    ++ra;
                }
            }
        }
        *reinterpret_cast<uint4 *>(a.Xs + (int64_t)e * 8) =
            make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
    }
}

// The same image one output row (n, i) per workgroup.  The s input rows it
// draws on are one contiguous NHWC range: it is read as aligned 16-byte chunks
// (all of a thread's loads in flight together) into LDS, then the row is
// written in 16-byte chunks.  Rows above or below the image are masked when
// read back, so whatever the range picks up there is never used.  Used when
// the range fits kS2dRowLds (the kernel above covers the rest).
constexpr int kS2dRowLds = 64 * 1024;

template <int NT>
__global__ __launch_bounds__(NT) void k_s2d_rows(S2dArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const int ni = blockIdx.x;  // (n, i)
    const int n = (int)fdiv((uint32_t)ni, a.divHs);
    const int i = ni - n * a.Hs;
    const int rowlen = a.W * a.Cx;
    const int h0 = i * a.s - a.pad;
    const int64_t b0 = ((int64_t)n * a.H + h0) * rowlen * 2;  // byte offset of (n, h0, 0, 0); may be < 0
    const int64_t a0 = b0 & ~(int64_t)15;
    const int nchunk = (int)((b0 - a0 + (int64_t)a.s * rowlen * 2 + 15) >> 4);
    const __amdgpu_buffer_rsrc_t xrs = rsrc(a.X, a.x_bytes);
    for (int base = 0; base < nchunk; base += 4 * NT) {
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int ch = base + u * NT + (int)threadIdx.x;
            const int64_t off = a0 + (int64_t)ch * 16;
            v[u] = bload16(xrs, (ch < nchunk && off >= 0 && off + 16 <= (int64_t)a.x_bytes) ? (uint32_t)off : kInvalidOffset);
            // the chunk that holds the input's last bytes (a buffer load reads
            // zero for a dword reaching past the range, and an odd element
            // count leaves the last dword half inside): its elements one by one
            if (ch < nchunk && off < (int64_t)a.x_bytes && off + 16 > (int64_t)a.x_bytes && off >= 0) {
                uint32_t w[4] = {0, 0, 0, 0};
                for (int q = 0; q < 8 && off + 2 * q < (int64_t)a.x_bytes; ++q)
                    w[q >> 1] |= (uint32_t)a.X[(off >> 1) + q] << (16 * (q & 1));
                v[u] = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int ch = base + u * NT + (int)threadIdx.x;
            if (ch < nchunk) reinterpret_cast<uint4 *>(smem)[ch] = v[u];
        }
    }
    __syncthreads();
    const uint16_t *rowbuf = reinterpret_cast<const uint16_t *>(smem) + (int)((b0 - a0) >> 1);
    uint16_t *dst = a.Xs + (int64_t)ni * a.Ws * a.Cs;
    if (a.runs) {
        // Cs = s*s*Cx and s*Cx*2 bytes a multiple of 8: output pixel j holds,
        // for each input row ra of the block, the s*Cx consecutive inputs
        // X[h0 + ra][j*s - pad ..][0 .. Cx) as one run of consecutive channels,
        // 8-byte aligned in the output; one thread per (j, ra) run
        const int run = a.s * a.Cx;
        for (int t = threadIdx.x; t < a.Ws * a.s; t += NT) {
            const int j = (int)fdiv((uint32_t)t, a.divS), ra = t - j * a.s;
            const int w0 = j * a.s - a.pad;
            const bool row_in = (unsigned)(h0 + ra) < (unsigned)a.H;
            const uint16_t *src = rowbuf + ra * rowlen + w0 * a.Cx;
            uint2 *out = reinterpret_cast<uint2 *>(dst + (int64_t)j * a.Cs + ra * run);
            const bool full = row_in && w0 >= 0 && w0 + a.s <= a.W;  // no zero padding in the run
            for (int q = 0; q < run; q += 4) {
                uint32_t v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (full) {
                        v[e] = src[q + e];
                    } else {  // a run at the image border: element by element
                        const int w = w0 + (q + e) / a.Cx;
                        v[e] = row_in && (unsigned)w < (unsigned)a.W ? src[q + e] : 0u;
                    }
                }
                out[q / 4] = make_uint2(v[0] | (v[1] << 16), v[2] | (v[3] << 16));
            }
        }
        return;
    }
    const int cs8 = a.Cs / 8;
    for (int e = threadIdx.x; e < a.Ws * cs8; e += NT) {
        const int j = (int)fdiv((uint32_t)e, a.divCs8);
        const int c0 = (e - j * cs8) * 8;
        int blk = (int)fdiv((uint32_t)c0, a.divCx);
        int c = c0 - blk * a.Cx;
        int ra = (int)fdiv((uint32_t)blk, a.divS);
        int rb = blk - ra * a.s;
        uint32_t v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int w = j * a.s + rb - a.pad;
            const bool in = c0 + q < a.Creal && (unsigned)(h0 + ra) < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
            v[q] = in ? rowbuf[ra * rowlen + w * a.Cx + c] : 0u;
            if (++c == a.Cx) {
                c = 0;
                if (++rb == a.s) {
                    rb = 0;
                    ++ra;
                }
            }
        }
        *reinterpret_cast<uint4 *>(dst + e * 8) =
            make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
    }
}

// ---------------------------------------------------------------- k_s2d_weights
// The compacted weights of a layer that runs on its space-to-depth image
// (factor s, Cx input channels, gD image taps per row, gCx image channels):
// column j (tap (kh, kw), input channel c) of row m moves to column
// (kh / s * gD + kw / s) * gCx + ((kh % s) * s + kw % s) * Cx + c of a row of
// ldk2; every other column is +0.  One workgroup per row, staged in LDS.
struct S2dWArgs {
    const uint16_t *Wc;
    const int32_t *col_ch, *col_tap;
    uint16_t *Ws;
    int32_t K, ldk, ldk2, D, s, Cx, gD, gCx;
};
__global__ __launch_bounds__(256) void k_s2d_weights(S2dWArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint16_t srow[];  // [ldk2]
    const int m = blockIdx.x, tid = threadIdx.x;
    for (int k = tid; k < a.ldk2; k += 256) srow[k] = 0;
    __syncthreads();
    for (int j = tid; j < a.K; j += 256) {
        const int t = a.col_tap[j], kh = t / a.D, kw = t - kh * a.D, c = a.col_ch[j];
        const int k2 = ((kh / a.s) * a.gD + kw / a.s) * a.gCx + ((kh % a.s) * a.s + kw % a.s) * a.Cx + c;
        srow[k2] = a.Wc[(int64_t)m * a.ldk + j];
    }
    __syncthreads();
    uint4 *dst = reinterpret_cast<uint4 *>(a.Ws + (int64_t)m * a.ldk2);
    const uint4 *src = reinterpret_cast<const uint4 *>(srow);
    for (int k = tid; k < a.ldk2 / 8; k += 256) dst[k] = src[k];
}

// ---------------------------------------------------------------- host side
// Raises a kernel's dynamic LDS limit to the full 160 KB, once per device.
int allow_full_lds(const void *kern) {
    static std::mutex mu;
    static std::set<std::pair<const void *, int>> done;
    int dev = 0;
    if (int rc = check_hip(hipGetDevice(&dev), "conv: current device")) return rc;
    std::lock_guard<std::mutex> lock(mu);
    if (done.count({kern, dev})) return SA_OK;
    if (int rc = check_hip(hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes),
                           "conv: set LDS size"))
        return rc;
    done.insert({kern, dev});
    return SA_OK;
}

template <int BM, int BN, int WN, int WM>
int launch_conv(ConvArgs a, hipStream_t stream) {
    using Cfg = ConvCfg<BM, BN, WN, WM>;
    // blocks of group i: [begin, begin + mtiles * ntiles), m-tiles fastest;
    // with split K, ksplit copies of that range, one per chunk of slices
    const int ntiles = (a.NPQ + BM - 1) / BM;
    int begin = 0;
    for (int i = 0; i < a.ngroups; ++i) {
        a.g[i].mtiles = (a.g[i].M + BN - 1) / BN;
        a.g[i].begin = begin;
        begin += a.g[i].mtiles * ntiles;
    }
    a.base_blocks = begin;
    a.nblocks = begin * std::max(1, a.ksplit);
    auto kern = a.ksplit > 1 ? k_conv<BM, BN, WN, WM, true> : k_conv<BM, BN, WN, WM, false>;
    if (int rc = allow_full_lds(reinterpret_cast<const void *>(kern))) return rc;
    hipLaunchKernelGGL(kern, dim3(a.nblocks), dim3(Cfg::NT), Cfg::lds, stream, a);
    return check_hip(hipGetLastError(), "k_conv");
}

// Tile shape of the direct kernel for groups of Ms filters over NPQ pixels:
// 0 = 128 x 128, 1 = 128 x 64 (pixels x filters; eight wavefronts, two
// workgroups per CU by LDS); *blocks receives the tile count.  The slowest CU runs
// ceil(tiles / CUs) tiles, and a 128 x 64 tile takes about 3/4 of the time of
// a 128 x 128 one (0.53-0.87 measured over the ResNet-50 and AlexNet layers,
// most near 0.75), so 128 x 64 tiles when 3 rounds of them cost no more than
// 4 rounds of 128 x 128 ones.
int direct_pick(const int *Ms, int n, int NPQ, int64_t *blocks) {
    int64_t t128 = 0, t64 = 0;
    for (int i = 0; i < n; ++i) {
        t128 += (Ms[i] + 127) / 128;
        t64 += (Ms[i] + 63) / 64;
    }
    const int64_t ptiles = (NPQ + 127) / 128, cus = device_cus();
    t128 *= ptiles;
    t64 *= ptiles;
    const int64_t r128 = (t128 + cus - 1) / cus, r64 = (t64 + cus - 1) / cus;
    if (3 * r64 <= 4 * r128) {
        *blocks = t64;
        return 1;
    }
    *blocks = t128;
    return 0;
}

// One launch for every group of a, in direct_pick's tile shape.  Eight
// wavefronts per 128-pixel tile (two rows of four, each 32 pixels by 32 or 64
// filters) keep 16 wavefronts per CU in flight to cover the operand latency:
// over 94 ResNet-50 layer runs they took 0.73-1.05x (15% less in sum) of the
// time of four-wavefront tiles of the same size; for groups of at most 32
// filters 128 x 64 tiles also beat 256 x 32 ones with four wavefronts (CIFAR
// 3x3 layer of 32 kept filters 12.6 -> 10.0 us, [256,256,3,3] at 10% kept
// 39.4 -> 30.9 us).
int run_conv(ConvArgs a, hipStream_t stream) {
    if (a.ngroups == 0) return SA_OK;
    for (int i = 0; i < a.ngroups; ++i)
        a.g[i].divRun = make_fastdiv((uint32_t)std::max(1, a.g[i].run));  // a group without columns has run 0
    a.divPQ = make_fastdiv((uint32_t)(a.P * a.Q));
    a.divCy = make_fastdiv((uint32_t)std::max(1, a.Cy));
    a.divQ = make_fastdiv((uint32_t)a.Q);
    a.divD = make_fastdiv((uint32_t)a.D);
    int Ms[SA_MAX_CONV_GROUPS];
    for (int i = 0; i < a.ngroups; ++i) Ms[i] = a.g[i].M;
    int64_t blocks;
    switch (direct_pick(Ms, a.ngroups, a.NPQ, &blocks)) {
        case 0: return launch_conv<128, 128, 4, 2>(a, stream);
        default: return launch_conv<128, 64, 4, 2>(a, stream);
    }
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
        if (int rc = allow_full_lds(reinterpret_cast<const void *>(k_im2col))) return rc;
        hipLaunchKernelGGL(k_im2col, dim3(blocks), dim3(kGatherThreads), (size_t)lds, stream, g);
        return check_hip(hipGetLastError(), "k_im2col");
    }
    const int64_t chunks = (int64_t)g.NPQ * (g.ldk / 8);
    const size_t tab = (size_t)g.ldk * 4;
    if (int rc = allow_full_lds(reinterpret_cast<const void *>(k_im2col_global))) return rc;
    hipLaunchKernelGGL(k_im2col_global, dim3((unsigned)std::min<int64_t>(8192, (chunks + 255) / 256)), dim3(256), tab,
                       stream, g);
    return check_hip(hipGetLastError(), "k_im2col_global");
}

// ---------------------------------------------------------------- planning
enum GroupPath { kSkip, kDirect, kPatch, kGather };

template <int TM, int TN, int NW = 4>
int launch_patch(PatchArgs a, int lds, hipStream_t stream) {
    using Cfg = PatchCfg<TM, TN, NW>;
    const int ntiles = (a.NPQ + Cfg::BMB - 1) / Cfg::BMB;
    int begin = 0;
    for (int i = 0; i < a.ngroups; ++i) {
        a.g[i].mtiles = (a.g[i].M + Cfg::BNB - 1) / Cfg::BNB;
        a.g[i].begin = begin;
        begin += a.g[i].mtiles * ntiles;
    }
    a.nblocks = begin;
    auto kern = k_conv_patch<TM, TN, NW>;
    if (int rc = allow_full_lds(reinterpret_cast<const void *>(kern))) return rc;
    hipLaunchKernelGGL(kern, dim3(a.nblocks), dim3(Cfg::NT), (size_t)lds, stream, a);
    return check_hip(hipGetLastError(), "k_conv_patch");
}

struct ConvPlan {
    int P, Q, NPQ, Cy;
    int path[SA_MAX_CONV_GROUPS];
    int pix_bytes[SA_MAX_CONV_GROUPS], nch[SA_MAX_CONV_GROUPS], ch_lo8[SA_MAX_CONV_GROUPS];
    int TM, TN, NW, patch_bytes, tab_bytes, lds;  // k_conv_patch launch (when any group takes it; NW wavefronts)
    // the direct groups run on k_ig (16-row filter tiles) instead of k_conv
    bool direct_ig;
    // split K (launches that would fill few CUs): chunks, and the binary32
    // partial sums [ksplit][part_stride] at byte part_off of the scratch
    int ksplit;
    int64_t part_stride;
    size_t part_off;
    // geometry the footprint kernel sees: the input itself, or (s2d = factor > 0)
    // its space-to-depth image, which then takes the first s2d_bytes of the scratch
    int s2d, gH, gW, gCx, gC, gD, gs, gpad;
    size_t s2d_bytes;
    // s2d_direct: a one-group layer on the space-to-depth image runs the direct
    // kernels over every tap x channel of that image (a stride-1, unpadded
    // gC x gD CONV of gCx channels), with its weights rewritten in that column
    // order ([M][s2d_ldk] bf16 at byte s2d_w_off of the scratch, +0 where the
    // image's tap / channel is no kept column); eff = the sizes those kernels see
    bool s2d_direct;
    size_t s2d_w_off;
    sa_compact_sizes eff;
    size_t ws_need;  // scratch: space-to-depth image, rewritten weights, then the two-phase groups' rows
};

constexpr int kPatchTMs[5] = {6, 4, 3, 2, 1};

const void *patch_kernel(int TM, int TN, int NW) {
    switch (TM * 100 + TN * 10 + NW) {
        case 616: return reinterpret_cast<const void *>(k_conv_patch<6, 1, 6>);
        case 416: return reinterpret_cast<const void *>(k_conv_patch<4, 1, 6>);
        case 614: return reinterpret_cast<const void *>(k_conv_patch<6, 1, 4>);
        case 624: return reinterpret_cast<const void *>(k_conv_patch<6, 2, 4>);
        case 414: return reinterpret_cast<const void *>(k_conv_patch<4, 1, 4>);
        case 424: return reinterpret_cast<const void *>(k_conv_patch<4, 2, 4>);
        case 314: return reinterpret_cast<const void *>(k_conv_patch<3, 1, 4>);
        case 324: return reinterpret_cast<const void *>(k_conv_patch<3, 2, 4>);
        case 214: return reinterpret_cast<const void *>(k_conv_patch<2, 1, 4>);
        case 224: return reinterpret_cast<const void *>(k_conv_patch<2, 2, 4>);
        case 114: return reinterpret_cast<const void *>(k_conv_patch<1, 1, 4>);
        case 124: return reinterpret_cast<const void *>(k_conv_patch<1, 2, 4>);
        default: return nullptr;
    }
}

// Workgroups of the footprint kernel <TM, TN, NW> with `lds` bytes of LDS that
// one CU holds at once (registers and LDS, as the runtime reports them),
// capped at 2 (the per-workgroup time model below is fitted for at most two);
// the LDS-only estimate when no GPU answers (a size query without a device).
int patch_per_cu(int TM, int TN, int NW, int lds) {
    const int by_lds = std::max(1, std::min(2, kLdsBytes / std::max(1, lds)));
    const void *kern = patch_kernel(TM, TN, NW);
    int dev = 0;
    if (!kern || hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return by_lds;
    }
    static std::mutex mu;
    static std::map<std::tuple<const void *, int, int>, int> cache;
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = cache.find({kern, lds, dev});
        if (it != cache.end()) return it->second;
    }
    int n = 0;
    if (allow_full_lds(kern) != SA_OK ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, 64 * NW, lds) != hipSuccess || n <= 0) {
        (void)hipGetLastError();
        clear_error();
        return by_lds;
    }
    n = std::min(n, 2);
    std::lock_guard<std::mutex> lock(mu);
    cache[{kern, lds, dev}] = n;
    return n;
}
constexpr int kPatchFixed = 9;  // per-workgroup footprint copy, in 32-filter-block units

int patch_lds(int TM, int TN, int patch_bytes, int tab_bytes, int NW = 4) {
    const int a_bytes = 2 * 32 * TM * kPatchRowA * 2;
    const int c_bytes = 32 * NW * TN * (32 * TM + 8) * 2;
    return std::max(patch_bytes + tab_bytes + a_bytes, c_bytes);
}

// Split K when every group takes the direct kernel (on the input, or on its
// gathered im2col rows), the launches leave CUs idle and the tiles are long
// (small batches): the 64-column slices are cut into ksplit chunks (at most 8,
// at most one workgroup per CU in all), each workgroup writes binary32
// partial sums, and k_splitk_sum adds them in chunk order.  (The footprint kernel is not split:
// each of its workgroups copies the whole input footprint, which then
// dominates; measured slower at batch 1.)
void split_plan(const sa_compact_sizes &s, ConvPlan *pl) {
    ConvPlan &p = *pl;
    p.ksplit = 1;
    int nd = 0, ng = 0, Md[SA_MAX_CONV_GROUPS], Mg[SA_MAX_CONV_GROUPS];
    int min_sl = 1 << 30;
    for (int g = 0; g < s.groups; ++g) {
        if (p.path[g] == kSkip) continue;
        if (p.path[g] == kPatch) return;
        if (p.path[g] == kDirect)
            Md[nd++] = s.M[g];
        else  // two-phase: the direct kernel over the gathered rows
            Mg[ng++] = s.M[g];
        min_sl = std::min(min_sl, s.ldk[g] / kBK);
    }
    if (nd + ng == 0) return;
    int64_t base = 0, b;
    if (nd > 0) {
        direct_pick(Md, nd, p.NPQ, &b);
        base += b;
    }
    if (ng > 0) {
        direct_pick(Mg, ng, p.NPQ, &b);
        base += b;
    }
    // the columns split over ks workgroups per tile only while the tiles
    // leave CUs idle (ks <= CUs / tiles: one workgroup per CU), and only when
    // the slices taken off each tile's serial loop pay for the split: about
    // 9.5 us for the partial sums and the summing pass against 0.46 us per
    // 64-column slice of a lone workgroup (measured at batch 1 over the
    // ResNet-50 and AlexNet layers), i.e. min_sl * (ks - 1) / ks > 20
    const int64_t cus = device_cus();
    if (base >= cus) return;
    const int64_t ks = std::min<int64_t>(8, cus / base);
    if (ks < 2 || (int64_t)min_sl * (ks - 1) <= 20 * ks) return;
    p.ksplit = (int)ks;
    p.part_stride = ((int64_t)p.NPQ * p.Cy + 3) / 4 * 4;
    p.part_off = (p.ws_need + 255) / 256 * 256;
    p.ws_need = p.part_off + ((size_t)p.ksplit * p.part_stride * 4 + 255) / 256 * 256;
}

// Kernel for the groups read straight from the NHWC input (measured on
// gfx950 over the ResNet-50 and AlexNet layers, in isolation and inside a
// block of layers whose inputs come cold from HBM): k_ig, whose filter tiles
// grow in steps of 16, for groups of at most 64 kept filters that k_conv's
// 64-filter tiles would pad by 15% or more, over 384-512 columns and at least
// 2^16 pixels (AlexNet's first layer of 48 kept filters on its space-to-depth
// image: 62 vs 68 us); the eight-wavefront k_conv tiles otherwise (k_ig was
// 3-25% slower on every other layer tried, among them ResNet-50's 1x1 layers
// of 38 and 77 kept filters and its first layer).  Not for split K over
// workgroups (small batches).
void direct_plan(const sa_compact_sizes &s, ConvPlan *pl) {
    ConvPlan &p = *pl;
    p.direct_ig = false;
    if (p.ksplit > 1) return;
    int Ms[SA_MAX_CONV_GROUPS], n = 0, maxK = 0, maxM = 0;
    int64_t fine = 0;
    for (int g = 0; g < s.groups; ++g) {
        if (p.path[g] != kDirect) continue;
        maxK = std::max(maxK, s.K[g]);
        maxM = std::max(maxM, s.M[g]);
        Ms[n++] = s.M[g];
        fine += (s.M[g] + 15) / 16 * 16;
    }
    if (n == 0) return;
    int64_t blocks;
    constexpr int kBN[2] = {128, 64};
    const int BN = kBN[direct_pick(Ms, n, p.NPQ, &blocks)];
    int64_t coarse = 0;
    for (int i = 0; i < n; ++i) coarse += (int64_t)(Ms[i] + BN - 1) / BN * BN;
    p.direct_ig = maxM <= 64 && coarse * 100 >= fine * 115 && maxK >= 384 && maxK <= 512 && p.NPQ >= (1 << 16);
}

// Validates the descriptor (beyond validate_conv) and chooses, per conv group,
// the direct kernel (columns are every tap of one run of channels), the
// LDS-footprint kernel, or the two-phase gather when the footprint of even the
// smallest pixel tile does not fit in LDS.
int conv_plan(const sa_conv_desc &d, ConvPlan *pl) {
    if (int rc = validate_conv(d)) return rc;
    const sa_compact_sizes &s = *d.sizes;
    const int64_t P = ((int64_t)d.H + 2 * d.pad - d.C) / d.stride + 1;
    const int64_t Q = ((int64_t)d.W + 2 * d.pad - d.D) / d.stride + 1;
    const int64_t NPQ = (int64_t)d.N * P * Q;
    if (d.Cx > 65535) return fail(SA_E_UNSUPPORTED, "conv: Cx > 65535");
    if ((int64_t)d.N * d.H * d.W * d.Cx * 2 >= (int64_t(1) << 31))
        return fail(SA_E_UNSUPPORTED, "conv: input of 2 GiB or more");
    ConvPlan &p = *pl;
    memset(&p, 0, sizeof p);
    p.NW = 4;
    p.P = (int)P;
    p.Q = (int)Q;
    p.NPQ = (int)NPQ;
    // pixels that are not whole 16-byte chunks (few input channels): the layer
    // runs on its space-to-depth image (s = stride; s = 1 only pads), whose
    // s*s*Cx channels are padded with zeros to a multiple of 8
    const int st = d.stride;
    p.s2d = 0;
    if (d.Cx % 8 != 0) {
        p.s2d = st;
        p.gH = (d.H + 2 * d.pad + st - 1) / st;
        p.gW = (d.W + 2 * d.pad + st - 1) / st;
        p.gCx = (d.Cx * st * st + 7) / 8 * 8;
        p.gC = (d.C + st - 1) / st;
        p.gD = (d.D + st - 1) / st;
        p.gs = 1;
        p.gpad = 0;
        p.s2d_bytes = (size_t)d.N * p.gH * p.gW * p.gCx * 2;
        if (p.s2d_bytes >= (size_t(1) << 31) || p.gCx > 65535) p.s2d = 0;  // too large: two-phase
    }
    if (p.s2d == 0) {
        p.gH = d.H;
        p.gW = d.W;
        p.gCx = d.Cx;
        p.gC = d.C;
        p.gD = d.D;
        p.gs = st;
        p.gpad = d.pad;
        p.s2d_bytes = 0;
    }
    // a one-group layer of at most 64 filters on its space-to-depth image: the
    // direct kernels read whole 16-byte chunks of the image's gCx channels at
    // each of its gC x gD taps, where the footprint kernel gathers 2-byte
    // columns from LDS (measured on the 7x7 and 11x11 stems: 38-48 filters
    // faster direct, 96 filters faster on the footprint kernel)
    p.s2d_direct = false;
    if (p.s2d > 0 && s.groups == 1 && s.M[0] > 0 && s.M[0] <= 64) {
        const int64_t K2 = (int64_t)p.gC * p.gD * p.gCx, ldk2 = (K2 + kBK - 1) / kBK * kBK;
        p.s2d_direct = K2 <= 16384 && ((int64_t)s.M[0] + 256) * ldk2 * 2 < (int64_t(1) << 31);
    }
    int max_ldk = 0, ngath = 0;
    for (int g = 0; g < s.groups; ++g) {
        if (s.ldk[g] != (s.K[g] + kBK - 1) / kBK * kBK || s.wc_offset[g] % 8 != 0)
            return fail(SA_E_ARG, "conv: sizes->ldk / wc_offset of group %d are not those of structadmm_compact", g);
        if (((int64_t)s.M[g] + 256) * s.ldk[g] * 2 >= (int64_t(1) << 31))
            return fail(SA_E_UNSUPPORTED, "conv: compacted matrix of group %d of 2 GiB or more", g);
        if (s.K[g] > 0 && (s.ch_lo[g] < 0 || s.ch_span[g] <= 0 || s.ch_lo[g] + s.ch_span[g] > d.Cx))
            return fail(SA_E_ARG, "conv: channel span of group %d outside the input's %d channels", g, d.Cx);
        p.Cy += s.M[g];
        if (s.M[g] == 0) {
            p.path[g] = kSkip;  // no output channels in this group
        } else if (p.s2d_direct || is_vec(s, g, d.Cx)) {
            p.path[g] = kDirect;
        } else {
            // the LDS copy is filled with 16-byte loads of 8 channels from an
            // 8-aligned channel window; inputs whose pixels are not a whole
            // number of such chunks (few input channels) gather their rows in a
            // separate pass instead
            p.path[g] = p.gCx % 8 == 0 ? kPatch : kGather;
            if (p.path[g] == kGather) continue;
            if (p.s2d > 0) {  // every channel of the space-to-depth pixel
                p.ch_lo8[g] = 0;
                p.nch[g] = p.gCx / 8;
            } else {
                const int lo = s.K[g] > 0 ? s.ch_lo[g] : 0;
                const int hi = s.K[g] > 0 ? s.ch_lo[g] + s.ch_span[g] : 1;
                p.ch_lo8[g] = lo / 8 * 8;
                p.nch[g] = (hi - p.ch_lo8[g] + 7) / 8;
            }
            // 16 bytes per chunk plus one word: an odd number of words per pixel,
            // so the lanes of an output row hit distinct banks
            const int bytes = p.nch[g] * 16 + 4;
            p.pix_bytes[g] = bytes;
            max_ldk = std::max(max_ldk, s.ldk[g]);
            ++ngath;
        }
    }
    if (ngath > 0) {
        // filter tile: least padded filter work; among those, the fewest
        // rounds of workgroups times the per-workgroup time, modelled (at 128
        // pixels per tile) as a fixed part for the footprint copy worth nine
        // 32-filter blocks (measured on the 13x13 AlexNet layers) plus one
        // unit per 32-filter block; TM >= 6 runs one workgroup per CU
        // (registers), smaller tiles up to two (LDS permitting)
        const int Hp = p.gH + 2 * p.gpad, Wp = p.gW + 2 * p.gpad;
        const int Ws = (Wp + p.gs - 1) / p.gs, Wpp = Ws * p.gs;
        p.tab_bytes = ((max_ldk + 2 * kPatchSlice) * 4 + 15) / 16 * 16;  // two slices past the last
        int64_t least = -1;
        for (int tm : kPatchTMs) {
            int64_t cost = 0;
            for (int g = 0; g < s.groups; ++g)
                if (p.path[g] == kPatch) cost += (s.M[g] + 32 * tm - 1) / (32 * tm) * (32 * tm);
            if (least < 0 || cost < least) least = cost;
        }
        const int rows128 = patch_rows(p.NPQ, p.P, p.Q, Hp, p.gs, p.gC, 128);
        int64_t pb128 = 0;
        for (int g = 0; g < s.groups; ++g)
            if (p.path[g] == kPatch)
                pb128 = std::max<int64_t>(pb128, ((int64_t)rows128 * Wpp * p.pix_bytes[g] + 15) / 16 * 16);
        int best_tm = 4;
        int64_t best_t = -1;
        for (int tm : kPatchTMs) {
            int64_t cost = 0, mt = 0;
            for (int g = 0; g < s.groups; ++g)
                if (p.path[g] == kPatch) {
                    cost += (s.M[g] + 32 * tm - 1) / (32 * tm) * (32 * tm);
                    mt += (s.M[g] + 32 * tm - 1) / (32 * tm);
                }
            if (cost != least) continue;
            const int64_t lds = pb128 <= kLdsBytes ? patch_lds(tm, 1, (int)pb128, p.tab_bytes) : kLdsBytes;
            const int64_t per_cu = patch_per_cu(tm, 1, 4, (int)lds);
            const int64_t wgs = mt * ((p.NPQ + 127) / 128);
            const int64_t t = (wgs + 256 * per_cu - 1) / (256 * per_cu) * (kPatchFixed + tm);
            if (best_t < 0 || t < best_t) best_t = t, best_tm = tm;
        }
        p.TM = best_tm;
        auto fits = [&](int tn, int *patch_bytes) {
            const int rows = patch_rows(p.NPQ, p.P, p.Q, Hp, p.gs, p.gC, 128 * tn);
            int64_t pb = 0;
            for (int g = 0; g < s.groups; ++g)
                if (p.path[g] == kPatch) pb = std::max<int64_t>(pb, ((int64_t)rows * Wpp * p.pix_bytes[g] + 15) / 16 * 16);
            if (pb > kLdsBytes) return false;
            *patch_bytes = (int)pb;
            return patch_lds(p.TM, tn, (int)pb, p.tab_bytes) <= kLdsBytes;
        };
        int64_t mt = 0;
        for (int g = 0; g < s.groups; ++g)
            if (p.path[g] == kPatch) mt += (s.M[g] + 32 * p.TM - 1) / (32 * p.TM);
        int pb2 = 0, pb1 = 0;
        const bool f2 = fits(2, &pb2), f1 = fits(1, &pb1);
        // two pixel fragments per wavefront halve the weight reads per MFMA, as
        // long as the launch still has two tiles per compute unit
        if (f2 && (!f1 || mt * ((p.NPQ + 255) / 256) >= 512)) {
            p.TN = 2;
            p.patch_bytes = pb2;
        } else if (f1) {
            p.TN = 1;
            p.patch_bytes = pb1;
        } else {
            p.TN = 0;
        }
        if (p.TN > 0) {
            p.lds = patch_lds(p.TM, p.TN, p.patch_bytes, p.tab_bytes);
            // six wavefronts (192-pixel tiles) when that saves rounds of workgroups
            // over the 256 CUs: a launch of one workgroup per CU whose last round
            // is partly filled (AlexNet conv4/conv5: 338 tiles) can take one round
            // fewer, each workgroup about 1.5 times as long
            if (p.TN == 1 && (p.TM == 6 || p.TM == 4)) {
                const int rows6 = patch_rows(p.NPQ, p.P, p.Q, Hp, p.gs, p.gC, 192);
                int64_t pb6 = 0;
                for (int g = 0; g < s.groups; ++g)
                    if (p.path[g] == kPatch) pb6 = std::max<int64_t>(pb6, ((int64_t)rows6 * Wpp * p.pix_bytes[g] + 15) / 16 * 16);
                const int64_t lds6 = pb6 <= kLdsBytes ? patch_lds(p.TM, 1, (int)pb6, p.tab_bytes, 6) : (int64_t)kLdsBytes + 1;
                if (lds6 <= kLdsBytes) {
                    const int64_t per4 = patch_per_cu(p.TM, 1, 4, p.lds);
                    const int64_t per6 = patch_per_cu(p.TM, 1, 6, (int)lds6);
                    const int64_t r4 = (mt * ((p.NPQ + 127) / 128) + 256 * per4 - 1) / (256 * per4);
                    const int64_t r6 = (mt * ((p.NPQ + 191) / 192) + 256 * per6 - 1) / (256 * per6);
                    if (r6 * 3 <= r4 * 2) {  // a tie goes to six wavefronts (measured faster on the 13x13 layers)
                        p.NW = 6;
                        p.patch_bytes = (int)pb6;
                        p.lds = (int)lds6;
                    }
                }
            }
        } else {
            for (int g = 0; g < s.groups; ++g)
                if (p.path[g] == kPatch) p.path[g] = kGather;
        }
    }
    bool any_patch = false;
    for (int g = 0; g < s.groups; ++g) any_patch = any_patch || p.path[g] == kPatch;
    if (!any_patch && !p.s2d_direct) p.s2d_bytes = 0;
    p.ws_need = (p.s2d_bytes + 255) / 256 * 256;
    p.eff = s;
    if (p.s2d_direct) {
        const int K2 = p.gC * p.gD * p.gCx, ldk2 = (K2 + kBK - 1) / kBK * kBK;
        p.eff.K[0] = K2;
        p.eff.ldk[0] = ldk2;
        p.eff.run[0] = p.gCx;
        p.eff.run_base[0] = 0;
        p.eff.ch_lo[0] = 0;
        p.eff.ch_span[0] = p.gCx;
        p.eff.kpad[0] = 0;
        p.eff.wc_offset[0] = 0;
        p.s2d_w_off = p.ws_need;
        p.ws_need += ((size_t)s.M[0] * ldk2 * 2 + 255) / 256 * 256;
    }
    for (int g = 0; g < s.groups; ++g) {
        if (p.path[g] != kGather) continue;
        const int64_t bytes = NPQ * s.ldk[g] * 2;
        if (bytes >= (int64_t(1) << 31))
            return fail(SA_E_UNSUPPORTED, "conv: gathered rows of group %d need 2 GiB or more", g);
        p.ws_need += ((size_t)bytes + 255) / 256 * 256;  // each gathered group has its own rows
    }
    split_plan(p.eff, &p);
    direct_plan(p.eff, &p);
    return SA_OK;
}

}  // namespace
}  // namespace sa

using namespace sa;

extern "C" size_t structadmm_conv_workspace(const sa_conv_desc *desc) {
    if (!desc) return 0;
    ConvPlan p;
    if (conv_plan(*desc, &p) != SA_OK) {
        clear_error();
        return 0;
    }
    return p.ws_need;
}

extern "C" int structadmm_conv_plan(const sa_conv_desc *desc, sa_conv_plan_info *info) {
    clear_error();
    if (!desc || !info) return fail(SA_E_ARG, "conv_plan: desc and info are required");
    ConvPlan p;
    if (int rc = conv_plan(*desc, &p)) return rc;
    const sa_compact_sizes &s = *desc->sizes;
    memset(info, 0, sizeof *info);
    info->groups = s.groups;
    info->ksplit = p.ksplit;
    info->space_to_depth = p.s2d;
    IgArgs ia;
    memset(&ia, 0, sizeof ia);
    ia.NPQ = p.NPQ;
    for (int g = 0; g < s.groups; ++g) {
        switch (p.path[g]) {
            case kSkip: info->path[g] = SA_CONV_NONE; break;
            case kDirect:
                info->path[g] = p.direct_ig ? SA_CONV_DIRECT_IG : SA_CONV_DIRECT;
                ia.g[ia.ngroups++].M = s.M[g];
                break;
            case kPatch: info->path[g] = SA_CONV_FOOTPRINT; break;
            default: info->path[g] = SA_CONV_GATHER; break;
        }
    }
    if (p.direct_ig && ia.ngroups > 0) {
        for (int g = 0, i = 0; g < s.groups; ++g)
            if (p.path[g] == kDirect) ia.g[i++].ldk = p.eff.ldk[g];
        const int t = ig_pick(ia);
        ig_tile_shape(t, &info->ig_tile[0], &info->ig_tile[1], &info->ig_tile[2]);
        info->ig_tile[3] = 1;
    }
    bool patch = false;
    for (int g = 0; g < s.groups; ++g) patch = patch || p.path[g] == kPatch;
    if (patch) {
        info->footprint_tile[0] = p.TM;
        info->footprint_tile[1] = p.TN;
        info->footprint_tile[2] = p.NW;
    }
    if (!patch && !p.s2d_direct) info->space_to_depth = 0;
    return SA_OK;
}

extern "C" int structadmm_conv_fwd(const sa_conv_desc *desc, hipStream_t stream) {
    clear_error();
    if (!desc) return fail(SA_E_ARG, "conv: desc is required");
    const sa_conv_desc &d = *desc;
    ConvPlan p;
    if (int rc = conv_plan(d, &p)) return rc;
    if (p.ws_need > 0) {
        if (!d.ws || d.ws_bytes < p.ws_need)
            return fail(SA_E_WORKSPACE, "conv: scratch of %zu bytes required (%zu given)", p.ws_need,
                        d.ws ? d.ws_bytes : 0);
        if (!aligned(d.ws, 256)) return fail(SA_E_ALIGN, "conv: scratch must be 256-byte aligned");
    }
    const sa_compact_sizes &s = *d.sizes;
    const int P = p.P, Q = p.Q, NPQ = p.NPQ;
    const uint32_t x_bytes = (uint32_t)((int64_t)d.N * d.H * d.W * d.Cx * 2);

    // groups read straight from the NHWC input share one launch, groups with
    // arbitrary columns a second (LDS footprint) and, when their footprint is
    // too large, a gather pass plus a third, 1x1 launch
    ConvArgs direct, gathered;
    PatchArgs pa;
    memset(&direct, 0, sizeof direct);
    memset(&gathered, 0, sizeof gathered);
    memset(&pa, 0, sizeof pa);
    direct.Y = gathered.Y = pa.Y = d.Y;
    direct.Cy = gathered.Cy = pa.Cy = p.Cy;
    direct.ldy = gathered.ldy = pa.ldy = d.ldy ? d.ldy : p.Cy;
    direct.ksplit = gathered.ksplit = p.ksplit;
    if (p.ksplit > 1) {
        direct.part = gathered.part = reinterpret_cast<float *>(static_cast<uint8_t *>(d.ws) + p.part_off);
        direct.part_stride = gathered.part_stride = p.part_stride;
    }
    direct.NPQ = gathered.NPQ = pa.NPQ = NPQ;
    direct.H = d.H;
    direct.W = d.W;
    direct.D = d.D;
    direct.stride = d.stride;
    direct.pad = d.pad;
    direct.P = P;
    direct.Q = Q;
    gathered.H = gathered.W = gathered.D = gathered.stride = gathered.P = gathered.Q = 1;
    gathered.pad = 0;
    pa.X = d.X;
    pa.x_bytes = x_bytes;
    if (p.s2d_bytes > 0) {  // the footprint kernel reads the space-to-depth image
        S2dArgs sa2;
        memset(&sa2, 0, sizeof sa2);
        sa2.X = d.X;
        sa2.Xs = static_cast<uint16_t *>(d.ws);
        sa2.N = d.N;
        sa2.H = d.H;
        sa2.W = d.W;
        sa2.Cx = d.Cx;
        sa2.s = p.s2d;
        sa2.pad = d.pad;
        sa2.Hs = p.gH;
        sa2.Ws = p.gW;
        sa2.Cs = p.gCx;
        sa2.Creal = d.Cx * p.s2d * p.s2d;
        sa2.chunks = (int32_t)(p.s2d_bytes / 16);
        sa2.divCs8 = make_fastdiv((uint32_t)(p.gCx / 8));
        sa2.divWs = make_fastdiv((uint32_t)p.gW);
        sa2.divHs = make_fastdiv((uint32_t)p.gH);
        sa2.divCx = make_fastdiv((uint32_t)d.Cx);
        sa2.divS = make_fastdiv((uint32_t)p.s2d);
        sa2.runs = sa2.Cs == sa2.Creal && (p.s2d * d.Cx * 2) % 8 == 0;
        sa2.x_bytes = x_bytes;
        const size_t rowbytes = (size_t)p.s2d * d.W * d.Cx * 2 + 32;  // the s rows plus alignment slack
        if (rowbytes <= (size_t)kS2dRowLds) {
            // 128 threads: up to 16 workgroups per CU, so that enough rows are in flight
            if (int rc = allow_full_lds(reinterpret_cast<const void *>(k_s2d_rows<128>))) return rc;
            hipLaunchKernelGGL(k_s2d_rows<128>, dim3(d.N * p.gH), dim3(128), rowbytes, stream, sa2);
        } else {
            hipLaunchKernelGGL(k_s2d, dim3((unsigned)std::min(16384, (sa2.chunks + 255) / 256)), dim3(256), 0, stream,
                               sa2);
        }
        if (int rc = check_hip(hipGetLastError(), "k_s2d")) return rc;
        pa.X = sa2.Xs;
        pa.x_bytes = (uint32_t)p.s2d_bytes;
    }
    const uint16_t *Ws2d = nullptr;  // the s2d_direct layer's rewritten weights
    if (p.s2d_direct) {
        S2dWArgs wa;
        wa.Wc = d.Wc + s.wc_offset[0];
        wa.col_ch = d.col_ch + s.col_offset[0];
        wa.col_tap = d.col_tap + s.col_offset[0];
        wa.Ws = reinterpret_cast<uint16_t *>(static_cast<uint8_t *>(d.ws) + p.s2d_w_off);
        wa.K = s.K[0];
        wa.ldk = s.ldk[0];
        wa.ldk2 = p.eff.ldk[0];
        wa.D = d.D;
        wa.s = p.s2d;
        wa.Cx = d.Cx;
        wa.gD = p.gD;
        wa.gCx = p.gCx;
        hipLaunchKernelGGL(k_s2d_weights, dim3(s.M[0]), dim3(256), (size_t)wa.ldk2 * 2, stream, wa);
        if (int rc = check_hip(hipGetLastError(), "k_s2d_weights")) return rc;
        Ws2d = wa.Ws;
        // the direct kernels see a stride-1, unpadded gC x gD CONV of the image
        direct.H = p.gH;
        direct.W = p.gW;
        direct.D = p.gD;
        direct.stride = 1;
        direct.pad = 0;
    }
    pa.N = d.N;
    pa.H = p.gH;
    pa.W = p.gW;
    pa.Cx = p.gCx;
    pa.C = p.gC;
    pa.D = p.gD;
    pa.stride = p.gs;
    pa.pad = p.gpad;
    pa.P = P;
    pa.Q = Q;
    pa.Hp = p.gH + 2 * p.gpad;
    pa.Wp = p.gW + 2 * p.gpad;
    pa.Ws = (pa.Wp + p.gs - 1) / p.gs;
    pa.Wpp = pa.Ws * p.gs;
    pa.patch_bytes = p.patch_bytes;
    pa.tab_bytes = p.tab_bytes;
    pa.s2d = p.s2d > 1 ? p.s2d : 1;  // factor 1: channel padding only, taps unchanged
    pa.Do = d.D;
    pa.Cxo = d.Cx;
    pa.divQ = make_fastdiv((uint32_t)Q);
    pa.divCy = make_fastdiv((uint32_t)std::max(1, p.Cy));
    pa.divP = make_fastdiv((uint32_t)P);
    pa.divHp = make_fastdiv((uint32_t)pa.Hp);
    pa.divD = make_fastdiv((uint32_t)p.gD);
    pa.divS = make_fastdiv((uint32_t)p.gs);
    pa.divDo = make_fastdiv((uint32_t)d.D);
    pa.divS2d = make_fastdiv((uint32_t)std::max(1, p.s2d));
    size_t ws_off = (p.s2d_bytes + 255) / 256 * 256;
    for (int g = 0; g < s.groups; ++g) {
        if (p.path[g] == kSkip) continue;
        if (p.path[g] == kPatch) {
            PatchGroup &G = pa.g[pa.ngroups++];
            G.Wc = d.Wc + s.wc_offset[g];
            G.col_ch = d.col_ch + s.col_offset[g];
            G.col_tap = d.col_tap + s.col_offset[g];
            G.M = s.M[g];
            G.K = s.K[g];
            G.ldk = s.ldk[g];
            G.o_off = s.row_offset[g];
            G.ch_lo = p.ch_lo8[g];
            G.nch = p.nch[g];
            G.pix_bytes = p.pix_bytes[g];
            G.divNch = make_fastdiv((uint32_t)G.nch);
            continue;
        }
        const bool vec = p.path[g] == kDirect;
        ConvArgs &a = vec ? direct : gathered;
        ConvGroup &G = a.g[a.ngroups++];
        G.Wc = d.Wc + s.wc_offset[g];
        G.M = s.M[g];
        G.ldk = s.ldk[g];
        G.o_off = s.row_offset[g];
        if (p.s2d_direct) {  // every tap x channel of the space-to-depth image
            G.Wc = Ws2d;
            G.ldk = p.eff.ldk[g];
            G.X = pa.X;
            G.x_bytes = pa.x_bytes;
            G.Cx = p.gCx;
            G.K = p.eff.K[g];
            G.run = p.gCx;
            G.run_base = 0;
            continue;
        }
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
    if (p.direct_ig && direct.ngroups > 0) {
        // ragged kept-filter counts over few columns: the 16-row MFMA kernel
        IgArgs ia;
        memset(&ia, 0, sizeof ia);
        ia.X = p.s2d_direct ? pa.X : d.X;
        ia.Y = d.Y;
        ia.x_bytes = p.s2d_direct ? pa.x_bytes : x_bytes;
        ia.yshift = (int)((reinterpret_cast<uintptr_t>(d.Y) >> 1) & 7);
        ia.H = direct.H;
        ia.W = direct.W;
        ia.Cx = p.s2d_direct ? p.gCx : d.Cx;
        ia.D = direct.D;
        ia.stride = direct.stride;
        ia.pad = direct.pad;
        ia.P = P;
        ia.Q = Q;
        ia.NPQ = NPQ;
        ia.Cy = p.Cy;
        ia.ldy = d.ldy ? d.ldy : p.Cy;
        ia.ngroups = direct.ngroups;
        for (int i = 0; i < direct.ngroups; ++i) {
            const ConvGroup &c = direct.g[i];
            IgGroup &G = ia.g[i];
            G.Wc = c.Wc;
            G.M = c.M;
            G.K = c.K;
            G.ldk = c.ldk;
            G.run = c.run;
            G.run_base = c.run_base;
            G.o_off = c.o_off;
        }
        if (int rc = ig_run(ia, -1, stream)) return rc;
    } else if (int rc = run_conv(direct, stream)) {
        return rc;
    }
    if (pa.ngroups > 0) {
        int rc = SA_OK;
        switch (p.TM * 100 + p.TN * 10 + p.NW) {
            case 616: rc = launch_patch<6, 1, 6>(pa, p.lds, stream); break;
            case 416: rc = launch_patch<4, 1, 6>(pa, p.lds, stream); break;
            case 614: rc = launch_patch<6, 1>(pa, p.lds, stream); break;
            case 624: rc = launch_patch<6, 2>(pa, p.lds, stream); break;
            case 414: rc = launch_patch<4, 1>(pa, p.lds, stream); break;
            case 424: rc = launch_patch<4, 2>(pa, p.lds, stream); break;
            case 314: rc = launch_patch<3, 1>(pa, p.lds, stream); break;
            case 324: rc = launch_patch<3, 2>(pa, p.lds, stream); break;
            case 214: rc = launch_patch<2, 1>(pa, p.lds, stream); break;
            case 224: rc = launch_patch<2, 2>(pa, p.lds, stream); break;
            case 114: rc = launch_patch<1, 1>(pa, p.lds, stream); break;
            case 124: rc = launch_patch<1, 2>(pa, p.lds, stream); break;
            default: return fail(SA_E_ARG, "conv: no tile shape for the gathered groups");
        }
        if (rc) return rc;
    }
    if (int rc = run_conv(gathered, stream)) return rc;
    if (p.ksplit > 1) {
        const int64_t total = (int64_t)NPQ * p.Cy;
        const int64_t blocks = (total + 1023) / 1024;
        hipLaunchKernelGGL(k_splitk_sum, dim3((unsigned)blocks), dim3(256), 0, stream,
                           static_cast<const float *>(direct.part), p.part_stride, p.ksplit, d.Y, total, p.Cy,
                           direct.ldy);
        return check_hip(hipGetLastError(), "k_splitk_sum");
    }
    return SA_OK;
}
