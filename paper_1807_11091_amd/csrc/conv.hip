// gfx950 implicit-GEMM CONV over the compacted weight matrix (Section 3:
// after row / column pruning the CONV is still a full GEMM, only smaller).
//
// Per conv group g the GEMM is  Y^T[m, npq] = sum_k Wc_g[m, k] * Xcol[npq, k]
// with npq = (n, p, q) the output pixel and k a kept (tap, channel) column.
// The im2col matrix Xcol is never materialised: each workgroup gathers its
// [BM x 64] slice of it from the NHWC input straight into LDS.
//   - MFMA v_mfma_f32_32x32x16_bf16: A operand = Wc rows (kept filters),
//     B operand = Xcol rows (output pixels), fp32 accumulators;
//   - LDS rows padded by 8 bf16 (16 B) so the 16-byte fragment reads of a
//     wavefront spread over all banks;
//   - register prefetch of the next 64-wide K slice while the MFMAs of the
//     current one run;
//   - VEC mode: the group's columns are every tap times one run of input
//     channels (filter / channel pruning), loaded as 16-byte vectors of 8
//     channels; GATHER mode: arbitrary (tap, channel) columns (shape
//     pruning), gathered per element through a column table held in LDS;
//   - workgroup ids are remapped so that each XCD (8 per MI355X, each with
//     its own L2) walks a contiguous range of output tiles.
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

constexpr int kBK = 64;           // K slice per LDS stage
constexpr int kLdsPad = 8;        // bf16 padding per LDS row
constexpr int kLdsRow = kBK + kLdsPad;
constexpr int kMaxGatherK = 8192; // column table entries held in LDS (GATHER mode)

struct ConvArgs {
    const uint16_t *X;
    const uint16_t *Wc;  // group base
    const int32_t *col_ch;   // group base
    const int32_t *col_tap;  // group base
    uint16_t *Y;
    int32_t H, W, Cx, D, stride, pad, P, Q, NPQ, Cy;
    int32_t M, K, ldk, run, run_base, o_off;
    int32_t mtiles, ntiles, nblocks;
    FastDiv divPQ, divQ;
};

template <int BM, int BN, int WN, int WM, bool GATHER>
__global__ __launch_bounds__(64 * WN * WM) void k_conv(ConvArgs a) {
    constexpr int NT = 64 * WN * WM;
    constexpr int TM = BN / WM / 32;   // 32-row m tiles per wavefront
    constexpr int TN = BM / WN / 32;   // 32-col npq tiles per wavefront
    constexpr int WROWS = BN * 8 / NT; // Wc 16-byte chunks per thread per stage
    constexpr int XROWS = BM * 8 / NT; // Xcol 16-byte chunks per thread per stage
    static_assert(TM >= 1 && TN >= 1 && WROWS >= 1 && XROWS >= 1, "tile shape");
    static_assert(NT % 8 == 0, "threads");

    __shared__ __attribute__((aligned(16))) uint16_t sW[BN * kLdsRow];
    __shared__ __attribute__((aligned(16))) uint16_t sX[BM * kLdsRow];
    extern __shared__ uint32_t s_tab[];  // GATHER: packed (c, d, channel) per column

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wn = wave % WN, wm = wave / WN;

    // XCD-aware tile order: hardware places workgroup i on XCD i % 8; give
    // each XCD a contiguous range of logical tiles (m tiles fastest).
    int bid = blockIdx.x;
    if ((a.nblocks & 7) == 0) bid = (bid & 7) * (a.nblocks >> 3) + (bid >> 3);
    const int mt = bid % a.mtiles, nt = bid / a.mtiles;
    const int m0 = mt * BN, n0 = nt * BM;

    if constexpr (GATHER) {
        for (int k = tid; k < a.K; k += NT) {
            const int t = a.col_tap[k];
            const int c = t / a.D, d = t - c * a.D;
            s_tab[k] = ((uint32_t)c << 24) | ((uint32_t)d << 16) | (uint32_t)a.col_ch[k];
        }
        __syncthreads();
    }

    // this thread's fixed 16-byte column chunk and rows
    const int kc = tid & 7;
    const int rbase = tid >> 3;
    int xh0[XROWS], xw0[XROWS], xpix[XROWS];  // pixel index of (n, 0, 0)
    bool xok[XROWS];
#pragma unroll
    for (int i = 0; i < XROWS; ++i) {
        const int npq = n0 + rbase + i * (NT / 8);
        xok[i] = npq < a.NPQ;
        const int nn = xok[i] ? (int)fdiv((uint32_t)npq, a.divPQ) : 0;
        const int rem = xok[i] ? npq - nn * a.P * a.Q : 0;
        const int p = (int)fdiv((uint32_t)rem, a.divQ);
        const int q = rem - p * a.Q;
        xh0[i] = p * a.stride - a.pad;
        xw0[i] = q * a.stride - a.pad;
        xpix[i] = nn * a.H * a.W;
    }

    uint4 wreg[WROWS], xreg[XROWS];
    const int nstages = (a.K + kBK - 1) / kBK;

    auto load_stage = [&](int s) {
        const int k = s * kBK + kc * 8;
#pragma unroll
        for (int i = 0; i < WROWS; ++i) {
            const int m = m0 + rbase + i * (NT / 8);
            if (m < a.M && k < a.ldk)
                wreg[i] = *reinterpret_cast<const uint4 *>(a.Wc + (int64_t)m * a.ldk + k);
            else
                wreg[i] = make_uint4(0, 0, 0, 0);
        }
        if constexpr (!GATHER) {
            // k = tap * run + ch; the 8 columns of a chunk share the tap
            int tap = 0, ch = 0, c = 0, d = 0;
            if (k < a.K) {
                tap = k / a.run;
                ch = k - tap * a.run;
                c = tap / a.D;
                d = tap - c * a.D;
            }
#pragma unroll
            for (int i = 0; i < XROWS; ++i) {
                const int h = xh0[i] + c, w = xw0[i] + d;
                if (xok[i] && k < a.K && h >= 0 && h < a.H && w >= 0 && w < a.W) {
                    const int64_t off = (int64_t)(xpix[i] + h * a.W + w) * a.Cx + a.run_base + ch;
                    xreg[i] = *reinterpret_cast<const uint4 *>(a.X + off);
                } else {
                    xreg[i] = make_uint4(0, 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < XROWS; ++i) {
                uint32_t v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    v[e] = 0;
                    const int ke = k + e;
                    if (xok[i] && ke < a.K) {
                        const uint32_t ent = s_tab[ke];
                        const int h = xh0[i] + (int)(ent >> 24);
                        const int w = xw0[i] + (int)((ent >> 16) & 255u);
                        const int ch = (int)(ent & 0xffffu);
                        if (h >= 0 && h < a.H && w >= 0 && w < a.W && ch < a.Cx)
                            v[e] = a.X[(int64_t)(xpix[i] + h * a.W + w) * a.Cx + ch];
                    }
                }
                xreg[i] = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16),
                                     v[6] | (v[7] << 16));
            }
        }
    };
    auto store_stage = [&]() {
#pragma unroll
        for (int i = 0; i < WROWS; ++i)
            *reinterpret_cast<uint4 *>(&sW[(rbase + i * (NT / 8)) * kLdsRow + kc * 8]) = wreg[i];
#pragma unroll
        for (int i = 0; i < XROWS; ++i)
            *reinterpret_cast<uint4 *>(&sX[(rbase + i * (NT / 8)) * kLdsRow + kc * 8]) = xreg[i];
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    load_stage(0);
    store_stage();
    __syncthreads();

    const int frow = lane & 31, fk = (lane >> 5) * 8;
    for (int s = 0; s < nstages; ++s) {
        if (s + 1 < nstages) load_stage(s + 1);
#pragma unroll
        for (int kk = 0; kk < kBK; kk += 16) {
            bf16x8 af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const bf16x8 *>(&sW[(wm * (BN / WM) + i * 32 + frow) * kLdsRow + kk + fk]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bfr[j] = *reinterpret_cast<const bf16x8 *>(&sX[(wn * (BM / WN) + j * 32 + frow) * kLdsRow + kk + fk]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
        if (s + 1 < nstages) {
            store_stage();
            __syncthreads();
        }
    }

    // epilogue: accumulator (i, j, r) holds m = .. + (r/4)*8 + (lane/32)*4 + r%4, npq = .. + lane%32
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int npq = n0 + wn * (BM / WN) + j * 32 + (lane & 31);
            if (npq >= a.NPQ) continue;
            uint16_t *yrow = a.Y + (int64_t)npq * a.Cy + a.o_off;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = m0 + wm * (BN / WM) + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                if (m < a.M) yrow[m] = f32_to_bf16_bits(acc[i][j][r]);
            }
        }
}

template <int BM, int BN, int WN, int WM>
int launch_conv(const ConvArgs &base, bool gather, hipStream_t stream) {
    ConvArgs a = base;
    a.mtiles = (a.M + BN - 1) / BN;
    a.ntiles = (a.NPQ + BM - 1) / BM;
    a.nblocks = a.mtiles * a.ntiles;
    constexpr int NT = 64 * WN * WM;
    if (gather) {
        size_t lds = sizeof(uint32_t) * (size_t)a.K;
        hipLaunchKernelGGL((k_conv<BM, BN, WN, WM, true>), dim3(a.nblocks), dim3(NT), lds, stream, a);
    } else {
        hipLaunchKernelGGL((k_conv<BM, BN, WN, WM, false>), dim3(a.nblocks), dim3(NT), 0, stream, a);
    }
    return check_hip(hipGetLastError(), "k_conv");
}

}  // namespace
}  // namespace sa

using namespace sa;

extern "C" int structadmm_conv_fwd(const sa_conv_desc *desc, hipStream_t stream) {
    clear_error();
    if (!desc) return fail(SA_E_ARG, "conv: desc is required");
    const sa_conv_desc &d = *desc;
    if (int rc = validate_conv(d)) return rc;
    const sa_compact_sizes &s = *d.sizes;
    const int P = (d.H + 2 * d.pad - d.C) / d.stride + 1;
    const int Q = (d.W + 2 * d.pad - d.D) / d.stride + 1;
    int Cy = 0;
    for (int g = 0; g < s.groups; ++g) Cy += s.M[g];
    for (int g = 0; g < s.groups; ++g) {
        if (s.ldk[g] != (s.K[g] + 7) / 8 * 8 || s.wc_offset[g] % 8 != 0)
            return fail(SA_E_ARG, "conv: sizes->ldk / wc_offset of group %d are not those of structadmm_compact", g);
        if (s.run[g] == 0 && s.K[g] > kMaxGatherK)
            return fail(SA_E_UNSUPPORTED, "conv: gathered group with K=%d > %d columns", s.K[g], kMaxGatherK);
        if (d.Cx > 65535) return fail(SA_E_UNSUPPORTED, "conv: Cx > 65535");
    }
    for (int g = 0; g < s.groups; ++g) {
        if (s.M[g] == 0) continue;  // no output channels in this group
        ConvArgs a;
        memset(&a, 0, sizeof a);
        a.X = d.X;
        a.Wc = d.Wc + s.wc_offset[g];
        a.col_ch = d.col_ch + s.col_offset[g];
        a.col_tap = d.col_tap + s.col_offset[g];
        a.Y = d.Y;
        a.H = d.H;
        a.W = d.W;
        a.Cx = d.Cx;
        a.D = d.D;
        a.stride = d.stride;
        a.pad = d.pad;
        a.P = P;
        a.Q = Q;
        a.NPQ = d.N * P * Q;
        a.Cy = Cy;
        a.M = s.M[g];
        a.K = s.K[g];
        a.ldk = s.ldk[g];
        a.run = s.run[g];
        a.run_base = s.run_base[g];
        a.o_off = s.row_offset[g];
        a.divPQ = make_fastdiv((uint32_t)(P * Q));
        a.divQ = make_fastdiv((uint32_t)Q);
        const bool vec = s.run[g] > 0 && s.run[g] % 8 == 0 && s.run_base[g] % 8 == 0 && d.Cx % 8 == 0;
        const bool gather = !vec;
        int rc;
        if (a.K == 0) {
            // no kept column: the output channels of this group are all zero;
            // the kernel writes them (every stage loads zeros)
        }
        if (a.M > 64)
            rc = launch_conv<128, 128, 2, 2>(a, gather, stream);
        else if (a.M > 32)
            rc = launch_conv<256, 64, 4, 1>(a, gather, stream);
        else
            rc = launch_conv<256, 32, 4, 1>(a, gather, stream);
        if (rc) return rc;
    }
    return SA_OK;
}
