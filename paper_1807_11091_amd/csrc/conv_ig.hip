// gfx950 implicit-GEMM CONV for conv groups whose compacted columns are every
// tap times one run of consecutive input channels: dense layers and filter- or
// channel-pruned ones (Section 3, "Combination of structured sparsities":
// filter pruning removes rows of the GEMM matrix, channel pruning removes the
// columns of a channel at every tap; what is left is a smaller full GEMM).
//
// Per conv group the GEMM is  Y^T[m, px] = sum_k Wc[m, k] * Xcol[px, k]  with
// px = (n, p, q) an output pixel and k = tap * run + ch a kept column.  A tile
// is BM = WM * MT * 16 filters by BP = (4 / WM) * NF * 16 pixels, computed by
// four wavefronts with v_mfma_f32_16x16x32_bf16 (A = 16 filters x 32 columns,
// B = 32 columns x 16 pixels, binary32 accumulation), so a pruned layer's
// kept-filter count pads only to a multiple of 16 rows.
//
//   * Persistent workgroups: the launch has as many workgroups as fit on the
//     GPU at once, and each walks one contiguous range of tiles (filter tiles
//     of a pixel range are neighbours; ranges follow the XCD order, so
//     neighbouring ranges share an L2).  Loads run as one stream across tile
//     boundaries: the next tile's first loads are in flight while the current
//     tile's output is written, which matters for the many layers whose tile
//     has only one or two 64-column slices (1x1 CONVs).
//   * B (pixels) goes straight from HBM / L2 into the MFMA operand registers:
//     lane l loads the 16 bytes of 8 consecutive channels of its pixel l % 16
//     for columns (l / 16) * 8 .. + 8 of a 32-column step, one raw buffer load
//     per pixel fragment; rows past the output and taps outside the image
//     read zero through an offset past the buffer.  Loads run three steps
//     ahead of the MFMAs in a ring of four register sets (a deeper ring,
//     eight sets, measured slower: its registers cost a wavefront per SIMD).  Nothing of B goes
//     through LDS: every wavefront owns its pixels, so LDS would only add a
//     write and a read of each byte.
//   * A (compacted weights, shared by the four wavefronts) is staged through
//     LDS in 64-column slices (the compacted rows are padded to a multiple of
//     64 columns with +0), two buffers, one barrier per slice; each slice is
//     loaded into registers one slice before it is written to LDS.  Rows of
//     144 bytes put the 8 lanes of each ds_read_b128 pass on distinct banks.
//   * Epilogue: the tile goes to an LDS region of its own as bf16 (round to
//     nearest even), then to Y with 16-byte stores.  A tile that holds whole
//     output rows is one contiguous range of Y, staged with Y's own row pitch;
//     otherwise each row is staged shifted so that its 16-byte chunks in LDS
//     line up with 16-byte chunks of Y, and only a row's first and last chunk
//     go out element by element.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <type_traits>

#include "conv_ig.h"
#include "sa_conv_device.h"
#include "sa_host.h"

namespace sa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kStage = 64;          // weight columns per LDS slice
constexpr int kARow = kStage + 8;   // LDS row pitch of a weight slice (bf16 elements)
constexpr int kLdsMax = 160 * 1024;

template <int MT, int NF, int WM>
struct IgCfg {
    static constexpr int WN = 4 / WM;
    static constexpr int BM = WM * MT * 16;  // filters per tile
    static constexpr int BP = WN * NF * 16;  // pixels per tile
    static constexpr int AR = (BM * 8 + kThreads - 1) / kThreads;  // 16-byte weight chunks per thread per slice
    static constexpr int CP = BM + 16;       // LDS row pitch of a shifted output row (bf16 elements)
    static constexpr int a_bytes = 2 * BM * kARow * 2;
    static constexpr int c_bytes = BP * CP * 2;
    static constexpr int lds = a_bytes + c_bytes;
    static_assert(WM == 1 || WM == 2 || WM == 4, "four wavefronts");
    static_assert(lds <= kLdsMax, "LDS");
};

// Where a tile sits: its conv group, first filter, first pixel and slices.
struct TilePos {
    int gi, m0, p0, nst;
};

template <int BM, int BP>
__device__ inline TilePos tile_pos(const IgArgs &a, int t) {
    int gi = 0;
    while (gi + 1 < a.ngroups && t >= a.g[gi + 1].begin) ++gi;
    const IgGroup &G = a.g[gi];
    const int lb = t - G.begin;
    const int pt = lb / G.mtiles;
    return TilePos{gi, (lb - pt * G.mtiles) * BM, pt * BP, G.ldk / kStage};
}

template <int MT, int NF, int WM>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void k_ig(IgArgs a) {
    using Cfg = IgCfg<MT, NF, WM>;
    constexpr int WN = Cfg::WN, BM = Cfg::BM, BP = Cfg::BP, AR = Cfg::AR, CP = Cfg::CP;

    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint16_t *sA = reinterpret_cast<uint16_t *>(smem);                 // [2][BM][kARow]
    uint16_t *sC = reinterpret_cast<uint16_t *>(smem + Cfg::a_bytes);  // [BP][CP] or [BP][Cy]

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave - wm * WN;
    const int kq = lane >> 4;  // 8-column chunk of a 32-column step this lane supplies

    // this workgroup's tiles [t_begin, t_end)
    const int wg = xcd_remap(blockIdx.x, gridDim.x);
    const int t_begin = (int)((int64_t)a.ntiles * wg / gridDim.x);
    const int t_end = (int)((int64_t)a.ntiles * (wg + 1) / gridDim.x);
    if (t_begin >= t_end) return;

    // ---- A stream: 64-column weight slices, tile after tile
    int tA = t_begin, stA = 0;
    TilePos pA = tile_pos<BM, BP>(a, tA);
    uint4 areg[AR];
    auto a_load = [&]() {  // loads slice stA of tile tA (nothing past the last tile)
        if (tA >= t_end) return;
        const IgGroup &G = a.g[pA.gi];
        const __amdgpu_buffer_rsrc_t wrs = rsrc(G.Wc, (uint32_t)G.M * (uint32_t)G.ldk * 2u);
#pragma unroll
        for (int i = 0; i < AR; ++i) {
            const int c = tid + i * kThreads;
            const int row = c >> 3, kc = c & 7;
            // rows past M read as zero through the buffer range
            const uint32_t off = ((uint32_t)(pA.m0 + row) * (uint32_t)G.ldk + stA * kStage + kc * 8) * 2u;
            areg[i] = bload16(wrs, c < BM * 8 ? off : kInvalidOffset);
        }
        if (++stA == pA.nst) {
            stA = 0;
            if (++tA < t_end) pA = tile_pos<BM, BP>(a, tA);
        }
    };
    auto a_store = [&](int buf) {
#pragma unroll
        for (int i = 0; i < AR; ++i) {
            const int c = tid + i * kThreads;
            if (c < BM * 8) *reinterpret_cast<uint4 *>(&sA[(buf * BM + (c >> 3)) * kARow + (c & 7) * 8]) = areg[i];
        }
    };

    // ---- B stream: 32-column steps, tile after tile.  State of the next step
    // to load: tile tB, step sB of nsB; this lane's pixel in each fragment
    // (hb, wb: top-left input position, pbase: element offset of
    // (n, hb, wb, run_base)), and its column k = tap * run + ch, tap = c*D + d,
    // with delta = (c * W + d) * Cx + ch the element offset from pbase.
    const __amdgpu_buffer_rsrc_t xrs = rsrc(a.X, a.x_bytes);
    int tB = t_begin, sB = 0, nsB = 0, runB = 8, KB = 0;
    int hb[NF], wb[NF], pbase[NF];
    int nk = 0, nch = 0, nc = 0, nd = 0, ndelta = 0;
    auto advance = [&](int by) {
        nk += by;
        nch += by;
        ndelta += by;
        while (nch >= runB) {  // run < 32: a step spans several taps
            nch -= runB;
            ndelta += a.Cx - runB;
            if (++nd == a.D) {
                nd = 0;
                ++nc;
                ndelta += (a.W - a.D) * a.Cx;
            }
        }
    };
    auto b_tile = [&]() {  // set-up for tile tB
        const TilePos P = tile_pos<BM, BP>(a, tB);
        const IgGroup &G = a.g[P.gi];
        nsB = 2 * P.nst;
        runB = G.run;
        KB = G.K;
#pragma unroll
        for (int j = 0; j < NF; ++j) {
            const int px = P.p0 + (wn * NF + j) * 16 + (lane & 15);
            const int pxc = min(px, a.NPQ - 1);
            const int n = (int)fdiv((uint32_t)pxc, a.divPQ);
            const int rem = pxc - n * a.P * a.Q;
            const int p = (int)fdiv((uint32_t)rem, a.divQ);
            const int q = rem - p * a.Q;
            const int h0 = p * a.stride - a.pad, w0 = q * a.stride - a.pad;
            pbase[j] = ((n * a.H + h0) * a.W + w0) * a.Cx + G.run_base;  // h0, w0 may be negative
            hb[j] = px < a.NPQ ? h0 : -(1 << 28);                       // rows past the output read nothing
            wb[j] = w0;
        }
        nk = nch = nc = nd = ndelta = 0;
        advance(kq * 8);
    };
    b_tile();
    uint4 b[4][NF];
    // loads the next step into ring slot SLOT (zero past the matrix; nothing past the last tile)
    auto b_load = [&](auto slot_c) {
        constexpr int SLOT = decltype(slot_c)::value;
        if (tB >= t_end) return;
        const bool kin = nk < KB;
#pragma unroll
        for (int j = 0; j < NF; ++j) {
            const int h = hb[j] + nc, w = wb[j] + nd;
            const bool in = kin && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
            b[SLOT][j] = bload16(xrs, in ? (uint32_t)(pbase[j] + ndelta) * 2u : kInvalidOffset);
        }
        if (++sB == nsB) {
            sB = 0;
            if (++tB < t_end) b_tile();
        } else {
            advance(32);
        }
    };

    f32x4 acc[MT][NF];
    auto zero_acc = [&]() {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NF; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    };
    // one 32-column step: MT weight fragments from LDS times NF pixel fragments
    auto compute = [&](auto slot_c, int buf, int kk) {
        constexpr int SLOT = decltype(slot_c)::value;
        const uint16_t *A = sA + (buf * BM + wm * MT * 16 + (lane & 15)) * kARow + kk + kq * 8;
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            const bf16x8 af = *reinterpret_cast<const bf16x8 *>(A + i * 16 * kARow);
#pragma unroll
            for (int j = 0; j < NF; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, __builtin_bit_cast(bf16x8, b[SLOT][j]),
                                                                   acc[i][j], 0, 0, 0);
        }
    };

    // ---- epilogue of tile t: accumulator (i, j) register r holds filter
    // i*16 + (lane/16)*4 + r, pixel j*16 + lane%16 of the wavefront's sub-tile
    auto epilogue = [&](int t) {
        const TilePos P = tile_pos<BM, BP>(a, t);
        const IgGroup &G = a.g[P.gi];
        const int rows = min(BP, a.NPQ - P.p0);
        // count results per row, then (the last channels of a row) +0 up to
        // the row's padded pitch
        const int count = min(BM, (G.o_off + G.M == a.Cy ? a.ldy - G.o_off : G.M) - P.m0);
        const bool whole = G.mtiles == 1 && G.M == a.Cy && a.yshift == 0 && a.ldy == a.Cy;
        const int64_t e_tile = (int64_t)P.p0 * a.ldy + G.o_off + P.m0;  // Y offset of the tile's (0, 0)
        // LDS position of output (pl, m): whole rows keep Y's pitch Cy, other
        // rows sit at pl * CP + shift(pl), shift = Y's misalignment of the row
        const int pitch = whole ? a.Cy : CP;
#pragma unroll
        for (int j = 0; j < NF; ++j) {
            const int pl = (wn * NF + j) * 16 + (lane & 15);
            const int sh = whole ? 0 : (int)((e_tile + (int64_t)pl * a.ldy + a.yshift) & 7);
            uint16_t *row = sC + pl * pitch + sh;
#pragma unroll
            for (int i = 0; i < MT; ++i) {
                const int ml = (wm * MT + i) * 16 + kq * 4;
                uint16_t o[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = f32_to_bf16_bits(acc[i][j][e]);  // round to nearest even
                if (ml >= count) continue;  // filters past the group (padding rows)
                stage_quad(row + ml, o, count - ml);  // a quad may straddle the end of the group
            }
        }
        __syncthreads();
        if (whole) {  // one contiguous range of Y: [p0 * Cy, (p0 + rows) * Cy)
            const int total = rows * a.Cy;
            uint16_t *base = a.Y + (int64_t)P.p0 * a.Cy;
            for (int c = tid; c * 8 < total; c += kThreads) {
                const int e0 = c * 8;
                const uint4 v = *reinterpret_cast<const uint4 *>(sC + e0);
                if (e0 + 8 <= total) {
                    nt_store16(base + e0, v);
                } else {
                    const uint16_t *s = sC + e0;
                    for (int q = 0; e0 + q < total; ++q) base[e0 + q] = s[q];
                }
            }
            return;
        }
        // row segments: 16-byte chunks of LDS line up with 16-byte chunks of Y
        constexpr int CPR = BM / 8 + 2;  // chunks a shifted row segment can touch
        for (int c = tid; c < rows * CPR; c += kThreads) {
            const int pl = c / CPR, ci = c - pl * CPR;
            const int64_t e0 = e_tile + (int64_t)pl * a.ldy;
            const int sh = (int)((e0 + a.yshift) & 7);
            const int lo = ci * 8 - sh;  // tile-row index of the chunk's first element
            if (lo >= count) continue;
            const uint16_t *s = sC + pl * CP + ci * 8;
            uint16_t *dst = a.Y + e0 + lo;
            if (lo >= 0 && lo + 8 <= count) {
                nt_store16(dst, *reinterpret_cast<const uint4 *>(s));
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    if (lo + q >= 0 && lo + q < count) dst[q] = s[q];
            }
        }
    };

    // compute stream: tile tC, slice stC of nstC
    int tC = t_begin, stC = 0, nstC = pA.nst;
    // end of a slice: the tile's output when it was the tile's last slice;
    // false when the workgroup is done
    auto end_slice = [&]() -> bool {
        if (++stC == nstC) {
            epilogue(tC);
            zero_acc();
            stC = 0;
            if (++tC >= t_end) return false;
            nstC = tile_pos<BM, BP>(a, tC).nst;
        }
        return true;
    };

    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    using S2 = std::integral_constant<int, 2>;
    using S3 = std::integral_constant<int, 3>;
    // one conv group, one filter tile and one 64-column slice: every tile
    // multiplies the same weights, which stay in LDS (both buffers) for good
    const bool a_res = a.ngroups == 1 && a.g[0].mtiles == 1 && a.g[0].ldk == kStage;
    zero_acc();
    a_load();
    b_load(S0{});
    b_load(S1{});
    b_load(S2{});
    a_store(0);
    if (a_res) a_store(1);
    else a_load();  // the next slice (of this tile or the next one)
    __syncthreads();
    // two slices (four steps) per iteration; slot (s mod 4) holds step s of the
    // stream.  The barrier after each slice also keeps one tile's output
    // staging from overwriting the previous tile's before it is stored.
    for (;;) {
        b_load(S3{});
        compute(S0{}, 0, 0);
        b_load(S0{});
        compute(S1{}, 0, 32);
        if (!end_slice()) break;
        if (!a_res) {
            a_store(1);
            a_load();
        }
        __syncthreads();
        b_load(S1{});
        compute(S2{}, 1, 0);
        b_load(S2{});
        compute(S3{}, 1, 32);
        if (!end_slice()) break;
        if (!a_res) {
            a_store(0);
            a_load();
        }
        __syncthreads();
    }
}

struct Tile {
    int MT, NF, WM;
};
// instantiated tile shapes (filters x pixels per workgroup = WM*MT*16 x (4/WM)*NF*16)
constexpr Tile kTiles[] = {{2, 2, 1}, {3, 2, 1}};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

template <int MT, int NF, int WM>
int launch(IgArgs a, hipStream_t stream) {
    using Cfg = IgCfg<MT, NF, WM>;
    auto kern = k_ig<MT, NF, WM>;
    // workgroups resident per CU for this kernel and its LDS (asked once)
    static std::mutex mu;
    static int per_cu = 0;
    {
        std::lock_guard<std::mutex> lock(mu);
        if (per_cu == 0) {
            if (Cfg::lds > 64 * 1024)
                if (int rc = check_hip(hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                                           hipFuncAttributeMaxDynamicSharedMemorySize, Cfg::lds),
                                       "conv_ig: set LDS size"))
                    return rc;
            int n = 0;
            if (int rc = check_hip(hipOccupancyMaxActiveBlocksPerMultiprocessor(
                                       &n, reinterpret_cast<const void *>(kern), kThreads, Cfg::lds),
                                   "conv_ig: occupancy"))
                return rc;
            per_cu = std::max(1, n);
        }
    }
    const int ptiles = (a.NPQ + Cfg::BP - 1) / Cfg::BP;
    int begin = 0;
    for (int i = 0; i < a.ngroups; ++i) {
        a.g[i].mtiles = (a.g[i].M + Cfg::BM - 1) / Cfg::BM;
        a.g[i].begin = begin;
        begin += a.g[i].mtiles * ptiles;
    }
    a.ntiles = begin;
    const int grid = std::min(a.ntiles, per_cu * device_cus());
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kThreads), Cfg::lds, stream, a);
    return check_hip(hipGetLastError(), "k_ig");
}

int launch_tile(int t, const IgArgs &a, hipStream_t stream) {
    switch (t) {
        case 0: return launch<2, 2, 1>(a, stream);
        case 1: return launch<3, 2, 1>(a, stream);
        default: return fail(SA_E_ARG, "conv_ig: no tile shape %d", t);
    }
}

}  // namespace

int device_cus() {
    static std::mutex mu;
    static int cus[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    std::lock_guard<std::mutex> lock(mu);
    if (cus[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cus[dev] = n;
    }
    return cus[dev];
}

// Tile shape for a launch: 32 or 48 filters, the one that covers every
// group's kept filters (the plan sends this kernel groups of at most 48 kept
// filters; a tile over whole output rows writes one contiguous range of Y).
int ig_pick(const IgArgs &a) {
    int maxM = 0;
    for (int i = 0; i < a.ngroups; ++i) maxM = std::max(maxM, (int)a.g[i].M);
    return maxM <= 32 ? 0 : 1;
}

int ig_run(IgArgs a, int tile, hipStream_t stream) {
    if (a.ngroups == 0) return SA_OK;
    for (int i = 0; i < a.ngroups; ++i) a.g[i].divRun = make_fastdiv((uint32_t)std::max(1, a.g[i].run));
    a.divPQ = make_fastdiv((uint32_t)(a.P * a.Q));
    a.divQ = make_fastdiv((uint32_t)a.Q);
    a.divD = make_fastdiv((uint32_t)a.D);
    a.divCy = make_fastdiv((uint32_t)std::max(1, a.Cy));
    if (tile < 0) tile = ig_pick(a);
    return launch_tile(tile, a, stream);
}

int ig_num_tiles() { return kNumTiles; }

void ig_tile_shape(int t, int *MT, int *NF, int *WM) {
    *MT = kTiles[t].MT;
    *NF = kTiles[t].NF;
    *WM = kTiles[t].WM;
}

}  // namespace sa
