// gfx950 path for non-structured (element-wise) pruning.  Section 3's
// non-structured set keeps an arbitrary pattern of weights, which leaves no
// smaller dense GEMM; Section 5 runs such layers on a CSR sparse library and
// finds little or no speedup.  This file gives that comparison on MI355X.
//
// structadmm_csr: the element-wise projection lists its kept weights in
//   ascending flat order a*B*C*D + j, which is already CSR order.
//   k_csr_from_kept splits each index into (row, column), rounds the value to
//   bf16 and writes the row pointers at the row boundaries.
// structadmm_conv_sparse_fwd: three launches.
//   k_csr_rowpad - one workgroup: every row's entry count rounded up to 8,
//                  exclusive scan -> padded row starts in the scratch;
//   k_csr_prep   - one wavefront per row: each entry's byte offset in the LDS
//                  copy of the input footprint (tap row, tap column, channel)
//                  and its value; rows are padded with zero entries so that
//                  the CONV walks whole groups of 8;
//   k_conv_csr   - a workgroup copies the input footprint of 64*TN output
//                  pixels into LDS (the conv group's channels, zero halo,
//                  columns de-interleaved by the stride so that the pixels of
//                  an output row read consecutive words at every tap), then
//                  its 8 wavefronts walk the rows of 64 filters (wavefront w
//                  takes rows w, w+8, ...).  Per 8 entries the offsets and
//                  values are uniform across the wavefront (scalar loads);
//                  each lane gathers its pixels' 8 inputs from LDS and adds 4
//                  packed bf16 dot products (v_dot2c_f32_bf16) to a binary32
//                  accumulator.  The outputs are staged through LDS for
//                  16-byte stores.
// Every kept weight costs one LDS gather per output pixel: a pattern of single
// weights has no dense tile for the matrix cores, and the LDS gather rate, not
// the ALUs or HBM, bounds the CONV.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>
#include <set>
#include <utility>

#include "sa_device.h"
#include "sa_host.h"
#include "structadmm.h"

namespace sa {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kSpLds = 160 * 1024;
constexpr int kSpRsrcWord3 = 0x00020000;   // raw buffer resource: 32-bit data, range checked
constexpr uint32_t kSpInvalid = 0x80000000u;  // past every buffer here: reads return zero
constexpr int64_t kSpMaxRows = 65536;
constexpr int64_t kSpMaxCols = int64_t(1) << 20;

__device__ inline __amdgpu_buffer_rsrc_t sp_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kSpRsrcWord3);
}

__device__ inline uint4 sp_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

// Workgroup ids reach the 8 XCDs round-robin; each XCD (own L2) gets one
// contiguous range of ids, so the filter blocks of a pixel tile, which copy
// the same footprint, run on one XCD.
__device__ inline int sp_xcd_remap(int bid, int n) {
    const int xcd = bid & 7, local = bid >> 3, q = n >> 3, r = n & 7;
    return xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

// ---------------------------------------------------------------- CSR build
struct CsrArgs {
    const float *Z;
    const int32_t *kept;
    int32_t *row_ptr;
    int32_t *col;
    uint16_t *val;
    int32_t A, K, nnz;
    uint32_t n;
    FastDiv divK;
};

// Thread e (0 <= e <= nnz) handles entry e and writes the row pointers of the
// rows that start at it: rows (row(e-1), row(e)] (thread nnz closes the rows
// after the last entry).  Indices past the tensor count as row A.
__global__ __launch_bounds__(256) void k_csr_from_kept(CsrArgs a) {
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e > a.nnz) return;
    auto row_of = [&](int i) {
        const uint32_t f = (uint32_t)a.kept[i];
        return f < a.n ? (int)fdiv(f, a.divK) : a.A;
    };
    const int prev = e == 0 ? -1 : row_of(e - 1);
    const int cur = e == a.nnz ? a.A : row_of(e);
    if (e < a.nnz) {
        const uint32_t f = (uint32_t)a.kept[e];
        int32_t c = 0;
        uint16_t v = 0;
        if (f < a.n) {
            c = (int32_t)(f - (uint32_t)cur * (uint32_t)a.K);
            v = f32_to_bf16_bits(a.Z[f]);
        }
        a.col[e] = c;
        a.val[e] = v;
    }
    for (int r = max(prev + 1, 0); r <= min(cur, a.A); ++r) a.row_ptr[r] = e;
}

// ---------------------------------------------------------------- CONV prep
// Row r's entries, clamped to [0, nnz): a row pointer array that is not
// monotone yields empty or shortened rows, never an access out of bounds.
__device__ inline void row_range(const int32_t *rp, int r, int nnz, int *lo, int *hi) {
    *lo = min(max(rp[r], 0), nnz);
    *hi = min(max(rp[r + 1], 0), nnz);
    if (*hi < *lo) *hi = *lo;
}

struct PadArgs {
    const int32_t *rp;
    int32_t *rowp8;
    int32_t A, nnz, cap;
};

__global__ __launch_bounds__(1024) void k_csr_rowpad(PadArgs a) {
    __shared__ uint32_t tmp[1024 / 64 + 1];
    uint32_t carry = 0;  // <= cap < 2^31; a block adds at most 1024 * 2^20
    for (int base = 0; base < a.A; base += 1024) {
        const int m = base + (int)threadIdx.x;
        uint32_t c = 0;
        if (m < a.A) {
            int lo, hi;
            row_range(a.rp, m, a.nnz, &lo, &hi);
            c = (uint32_t)(hi - lo + 7) & ~7u;
        }
        uint32_t total;
        const uint32_t ex = block_excl_scan(c, tmp, &total);
        if (m < a.A) a.rowp8[m] = (int32_t)min(carry + ex, (uint32_t)a.cap);
        carry = min(carry + total, (uint32_t)a.cap);
    }
    if (threadIdx.x == 0) a.rowp8[a.A] = (int32_t)carry;
}

struct PrepArgs {
    const int32_t *rp;
    const int32_t *col;
    const uint16_t *val;
    const int32_t *rowp8;
    int32_t *off8;
    uint16_t *val8;
    int32_t A, nnz, K, CD, D, B, stride, Ws, rowb, pixb;
    FastDiv divCD, divD, divS, divPG;
};

__global__ __launch_bounds__(256) void k_csr_prep(PrepArgs a) {
    const int m = blockIdx.x * 4 + (int)(threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (m >= a.A) return;
    int lo, hi;
    row_range(a.rp, m, a.nnz, &lo, &hi);
    const int s0 = a.rowp8[m], s1 = a.rowp8[m + 1];
    const int gc = (int)fdiv((uint32_t)m, a.divPG);
    const int ch0 = gc * a.B - (gc * a.B) / 8 * 8;  // channel b = 0 within the group's 8-aligned copy
    for (int t = lane; t < s1 - s0; t += 64) {
        int32_t o = 0;
        uint16_t v = 0;
        if (t < hi - lo) {
            const int j = a.col[lo + t];
            if ((unsigned)j < (unsigned)a.K) {
                const int b = (int)fdiv((uint32_t)j, a.divCD), tap = j - b * a.CD;
                const int c = (int)fdiv((uint32_t)tap, a.divD), d = tap - c * a.D;
                const int dq = (int)fdiv((uint32_t)d, a.divS), dr = d - dq * a.stride;
                o = c * a.rowb + (dr * a.Ws + dq) * a.pixb + (ch0 + b) * 2;
                v = a.val[lo + t];
            }
        }
        a.off8[s0 + t] = o;
        a.val8[s0 + t] = v;
    }
}

// ---------------------------------------------------------------- k_conv_csr
struct SpConvArgs {
    const uint16_t *X;
    uint16_t *Y;
    const int32_t *rowp8;
    const int32_t *off8;
    const uint16_t *val8;
    uint32_t x_bytes;
    int32_t N, H, W, Cx, A, B, C, stride, pad, P, Q, NPQ;
    int32_t Hp, Wp, Ws, Wpp, nch, pixb, rowb;
    int32_t per_group, fb_per_group, nfb, nblocks;
    FastDiv divQ, divP, divHp, divS, divFbg, divNch, divRowc;
};

template <int TN, int NW, int RPW>
__global__ __launch_bounds__(64 * NW) void k_conv_csr(SpConvArgs a) {
    constexpr int kSpThreads = 64 * NW, kSpWaves = NW;
    constexpr int kSpRowsPerWave = RPW;         // filter rows per wavefront
    constexpr int kSpFB = kSpRowsPerWave * NW;  // filters per workgroup (a multiple of 8)
    constexpr int kSpOutRow = kSpFB + 8;        // LDS row of the staged output tile (bf16 elements)
    constexpr int BP = 64 * TN;  // output pixels per workgroup
    constexpr int kUn = 8;       // 16-byte loads in flight per thread during the copy
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    const int bid = sp_xcd_remap(blockIdx.x, a.nblocks);
    const int tile = bid / a.nfb, fbi = bid - tile * a.nfb;
    const int gc = (int)fdiv((uint32_t)fbi, a.divFbg), fb = fbi - gc * a.fb_per_group;
    const int f0 = gc * a.per_group + fb * kSpFB;
    const int f1 = min(f0 + kSpFB, (gc + 1) * a.per_group);
    const int n0 = tile * BP;

    // 1. input footprint: padded rows [g0, g1) of the stacked padded images,
    //    channels [lo8, lo8 + 8*nch) (chunks past Cx read as zero)
    const int r0 = (int)fdiv((uint32_t)n0, a.divQ);
    const int r1 = (int)fdiv((uint32_t)(min(n0 + BP, a.NPQ) - 1), a.divQ);
    const int i0 = (int)fdiv((uint32_t)r0, a.divP), i1 = (int)fdiv((uint32_t)r1, a.divP);
    const int g0 = i0 * a.Hp + (r0 - i0 * a.P) * a.stride;
    const int g1 = i1 * a.Hp + (r1 - i1 * a.P) * a.stride + a.C;
    const int lo8 = (gc * a.B) / 8 * 8;
    const int rowc = a.Wp * a.nch;
    const int total = (g1 - g0) * rowc;
    const __amdgpu_buffer_rsrc_t xrs = sp_rsrc(a.X, a.x_bytes);
    for (int base = tid; base < total; base += kSpThreads * kUn) {
        uint4 v[kUn];
        int dst[kUn];
#pragma unroll
        for (int u = 0; u < kUn; ++u) {
            const int idx = base + u * kSpThreads;
            dst[u] = -1;
            uint32_t off = kSpInvalid;
            if (idx < total) {
                const int pr = (int)fdiv((uint32_t)idx, a.divRowc);
                const int rem = idx - pr * rowc;
                const int wpad = (int)fdiv((uint32_t)rem, a.divNch);
                const int ch = rem - wpad * a.nch;
                const int gr = g0 + pr;
                const int img = (int)fdiv((uint32_t)gr, a.divHp);
                const int h = gr - img * a.Hp - a.pad, w = wpad - a.pad;
                const int jw = (int)fdiv((uint32_t)wpad, a.divS);
                dst[u] = pr * a.rowb + ((wpad - jw * a.stride) * a.Ws + jw) * a.pixb + ch * 16;
                const int chan = lo8 + ch * 8;
                if (img < a.N && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W && chan < a.Cx)
                    off = ((((uint32_t)(img * a.H + h) * a.W + w) * a.Cx) + chan) * 2u;
            }
            v[u] = sp_load16(xrs, off);
        }
#pragma unroll
        for (int u = 0; u < kUn; ++u) {
            if (dst[u] < 0) continue;
            uint32_t *d32 = reinterpret_cast<uint32_t *>(smem + dst[u]);
            d32[0] = v[u].x;
            d32[1] = v[u].y;
            d32[2] = v[u].z;
            d32[3] = v[u].w;
        }
    }

    // byte offset of each pixel's window corner in the copy
    int pbase[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int px = n0 + j * 64 + lane;
        pbase[j] = 0;  // pixels past the output read the copy's first word; never stored
        if (px < a.NPQ) {
            const int r = (int)fdiv((uint32_t)px, a.divQ);
            const int img = (int)fdiv((uint32_t)r, a.divP);
            const int gr = img * a.Hp + (r - img * a.P) * a.stride;
            pbase[j] = (gr - g0) * a.rowb + (px - r * a.Q) * a.pixb;
        }
    }
    __syncthreads();

    // 2. rows f0 + wave + 8i: 8 entries at a time, uniform offsets and values
    uint16_t out[kSpRowsPerWave][TN];
#pragma unroll
    for (int i = 0; i < kSpRowsPerWave; ++i) {
        const int m = f0 + wave + kSpWaves * i;
        float acc[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[j] = 0.0f;
        if (m < f1) {
            const int e0 = __builtin_amdgcn_readfirstlane(a.rowp8[m]);
            const int e1 = __builtin_amdgcn_readfirstlane(a.rowp8[m + 1]);
            for (int e = e0; e < e1; e += 8) {
                const int4 oa = *reinterpret_cast<const int4 *>(a.off8 + e);
                const int4 ob = *reinterpret_cast<const int4 *>(a.off8 + e + 4);
                const uint4 wv = *reinterpret_cast<const uint4 *>(a.val8 + e);
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const uint8_t *pp = smem + pbase[j];
                    auto ld = [&](int o) { return (uint32_t)*reinterpret_cast<const uint16_t *>(pp + o); };
                    const uint32_t x0 = ld(oa.x) | (ld(oa.y) << 16);
                    const uint32_t x1 = ld(oa.z) | (ld(oa.w) << 16);
                    const uint32_t x2 = ld(ob.x) | (ld(ob.y) << 16);
                    const uint32_t x3 = ld(ob.z) | (ld(ob.w) << 16);
                    float s = acc[j];
                    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, x0),
                                                         __builtin_bit_cast(bf16x2, wv.x), s, false);
                    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, x1),
                                                         __builtin_bit_cast(bf16x2, wv.y), s, false);
                    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, x2),
                                                         __builtin_bit_cast(bf16x2, wv.z), s, false);
                    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, x3),
                                                         __builtin_bit_cast(bf16x2, wv.w), s, false);
                    acc[j] = s;
                }
            }
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) out[i][j] = f32_to_bf16_bits(acc[j]);
    }
    __syncthreads();  // the footprint is dead: the output tile reuses its LDS

    // 3. output tile [BP][kSpOutRow] through LDS, 16-byte stores of each pixel's filters
    uint16_t *sC = reinterpret_cast<uint16_t *>(smem);
#pragma unroll
    for (int i = 0; i < kSpRowsPerWave; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) sC[(j * 64 + lane) * kSpOutRow + wave + kSpWaves * i] = out[i][j];
    __syncthreads();
    constexpr int CPR = kSpFB / 8;
    for (int c = tid; c < BP * CPR; c += kSpThreads) {
        const int pl = c / CPR, mc = c - pl * CPR;
        const int px = n0 + pl, m = f0 + mc * 8;
        if (px >= a.NPQ || m >= f1) continue;
        uint16_t *dst = a.Y + (int64_t)px * a.A + m;
        const uint16_t *src = &sC[pl * kSpOutRow + mc * 8];
        const int n = min(8, f1 - m);
        if (n == 8 && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
            *reinterpret_cast<uint4 *>(dst) = *reinterpret_cast<const uint4 *>(src);
        } else {
            for (int q = 0; q < n; ++q) dst[q] = src[q];
        }
    }
}

// ---------------------------------------------------------------- host side
int sp_allow_full_lds(const void *kern) {
    static std::mutex mu;
    static std::set<std::pair<const void *, int>> done;
    int dev = 0;
    if (int rc = check_hip(hipGetDevice(&dev), "conv_sparse: current device")) return rc;
    std::lock_guard<std::mutex> lock(mu);
    if (done.count({kern, dev})) return SA_OK;
    if (int rc = check_hip(hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, kSpLds),
                           "conv_sparse: set LDS size"))
        return rc;
    done.insert({kern, dev});
    return SA_OK;
}

// Most padded input rows any tile of bp consecutive output pixels spans.
int sp_patch_rows(int NPQ, int P, int Q, int Hp, int stride, int C, int bp) {
    int best = 0;
    for (int n0 = 0; n0 < NPQ; n0 += bp) {
        const int r0 = n0 / Q, r1 = (std::min(n0 + bp, NPQ) - 1) / Q;
        const int g0 = (r0 / P) * Hp + (r0 % P) * stride;
        const int g1 = (r1 / P) * Hp + (r1 % P) * stride + C;
        best = std::max(best, g1 - g0);
    }
    return best;
}

// launch shapes in order of preference (see sp_plan)
struct SpShape {
    int tn, nw, rpw;
};
constexpr SpShape kSpShapes[] = {{2, 16, 8}, {1, 16, 8}, {2, 8, 8}, {1, 8, 8}, {1, 16, 1}, {1, 8, 1}};

struct SpPlan {
    int P, Q, NPQ, Hp, Wp, Ws, Wpp, nch, pixb, rowb, TN, NW, RPW, lds;
    int64_t cap;  // padded entries: nnz + 7 per row
    size_t off_at, val_at, ws_need;
};

int sp_plan(const sa_sparse_conv_desc &d, SpPlan *p) {
    if (d.N <= 0 || d.H <= 0 || d.W <= 0 || d.Cx <= 0 || d.A <= 0 || d.B <= 0 || d.C <= 0 || d.D <= 0 ||
        d.groups <= 0 || d.stride <= 0 || d.pad < 0)
        return fail(SA_E_ARG, "conv_sparse: sizes, groups and stride must be positive and pad >= 0");
    if (d.A % d.groups != 0 || (int64_t)d.groups * d.B != d.Cx)
        return fail(SA_E_ARG, "conv_sparse: need A %% groups == 0 and Cx == groups * B (A=%d B=%d groups=%d Cx=%d)",
                    d.A, d.B, d.groups, d.Cx);
    const int64_t K = (int64_t)d.B * d.C * d.D;
    if (d.nnz < 0 || d.nnz > (int64_t)d.A * K)
        return fail(SA_E_ARG, "conv_sparse: nnz=%lld outside [0, A*B*C*D]", (long long)d.nnz);
    if (d.A > kSpMaxRows || K > kSpMaxCols)
        return fail(SA_E_UNSUPPORTED, "conv_sparse: A <= %lld and B*C*D <= %lld supported", (long long)kSpMaxRows,
                    (long long)kSpMaxCols);
    if (d.Cx % 8 != 0)
        return fail(SA_E_UNSUPPORTED, "conv_sparse: input channels Cx=%d must be a multiple of 8", d.Cx);
    if (d.H + 2 * d.pad < d.C || d.W + 2 * d.pad < d.D)
        return fail(SA_E_ARG, "conv_sparse: output would be empty");
    p->P = (d.H + 2 * d.pad - d.C) / d.stride + 1;
    p->Q = (d.W + 2 * d.pad - d.D) / d.stride + 1;
    const int64_t NPQ = (int64_t)d.N * p->P * p->Q;
    if (NPQ >= (int64_t(1) << 31) || NPQ * d.A >= (int64_t(1) << 40))
        return fail(SA_E_UNSUPPORTED, "conv_sparse: output too large");
    if ((int64_t)d.N * d.H * d.W * d.Cx * 2 >= (int64_t(1) << 31))
        return fail(SA_E_UNSUPPORTED, "conv_sparse: input of 2 GiB or more");
    p->NPQ = (int)NPQ;
    p->Hp = d.H + 2 * d.pad;
    p->Wp = d.W + 2 * d.pad;
    p->Ws = (p->Wp + d.stride - 1) / d.stride;
    p->Wpp = p->Ws * d.stride;
    int nch = 0;
    for (int gc = 0; gc < d.groups; ++gc) {
        const int lo8 = gc * d.B / 8 * 8;
        nch = std::max(nch, (gc * d.B + d.B - lo8 + 7) / 8);
    }
    p->nch = nch;
    p->pixb = nch * 16 + 4;  // an odd number of words: the lanes of an output row hit distinct banks
    // rows of the copy are padded so that, at stride 1, pixel (r, q) of an image
    // starts at a bank given by its linear index r*Q + q: 64 consecutive output
    // pixels then hit 64 distinct banks across row ends as well
    const int pixw = p->pixb / 4;
    const int padw = d.stride == 1 ? (((p->Q - p->Wpp) * pixw) % 64 + 64) % 64 : 0;
    p->rowb = p->Wpp * p->pixb + 4 * padw;
    // launch shape: 64*TN pixels per workgroup, NW wavefronts of RPW filter
    // rows each.  First choice: two pixels per lane, 16 wavefronts of 8 rows
    // (more wavefronts to issue gathers, fewer footprint copies), as long as
    // the grid holds 512 workgroups; small layers (batch 1) take the shape
    // with the most workgroups, down to one row per wavefront
    const int per_group = d.A / d.groups;
    p->TN = 0;
    int64_t best_grid = -1;
    for (const SpShape &c : kSpShapes) {
        const int fb = c.nw * c.rpw;
        if (c.nw == 16 && c.rpw == 8 && per_group <= 64) continue;
        const int64_t rows = sp_patch_rows(p->NPQ, p->P, p->Q, p->Hp, d.stride, d.C, 64 * c.tn);
        const int64_t patch = (rows * p->rowb + 15) / 16 * 16;
        const int64_t lds = std::max<int64_t>(patch, (int64_t)64 * c.tn * (fb + 8) * 2);
        if (lds > kSpLds) continue;
        const int64_t grid = (p->NPQ + 64 * c.tn - 1) / (64 * c.tn) * d.groups * ((per_group + fb - 1) / fb);
        if (grid > best_grid) {
            best_grid = grid;
            p->TN = c.tn;
            p->NW = c.nw;
            p->RPW = c.rpw;
            p->lds = (int)lds;
        }
        if (grid >= 512) break;
    }
    if (p->TN == 0)
        return fail(SA_E_UNSUPPORTED, "conv_sparse: the input footprint of 64 output pixels exceeds LDS");
    p->cap = round_up(d.nnz + 7 * (int64_t)d.A, 8);  // every padded row start is a multiple of 8
    if (p->cap >= (int64_t(1) << 31))
        return fail(SA_E_UNSUPPORTED, "conv_sparse: too many entries");
    p->off_at = round_up(((size_t)d.A + 1) * 4, 256);
    p->val_at = p->off_at + round_up((size_t)p->cap * 4, 256);
    p->ws_need = p->val_at + round_up((size_t)p->cap * 2, 256);
    return SA_OK;
}

template <int TN, int NW, int RPW>
int launch_conv_csr(SpConvArgs a, int lds, hipStream_t stream) {
    auto kern = k_conv_csr<TN, NW, RPW>;
    if (int rc = sp_allow_full_lds(reinterpret_cast<const void *>(kern))) return rc;
    hipLaunchKernelGGL(kern, dim3(a.nblocks), dim3(64 * NW), (size_t)lds, stream, a);
    return check_hip(hipGetLastError(), "k_conv_csr");
}

// Padded row starts, entry offsets and values for the layer's CSR and geometry.
int sp_prepare(const sa_sparse_conv_desc &d, const SpPlan &p, int32_t *rowp8, int32_t *off8, uint16_t *val8,
               hipStream_t stream) {
    PadArgs pa;
    pa.rp = d.row_ptr;
    pa.rowp8 = rowp8;
    pa.A = d.A;
    pa.nnz = (int32_t)d.nnz;
    pa.cap = (int32_t)p.cap;
    hipLaunchKernelGGL(k_csr_rowpad, dim3(1), dim3(1024), 0, stream, pa);
    if (int rc = check_hip(hipGetLastError(), "k_csr_rowpad")) return rc;

    PrepArgs pr;
    pr.rp = d.row_ptr;
    pr.col = d.col;
    pr.val = d.val;
    pr.rowp8 = rowp8;
    pr.off8 = off8;
    pr.val8 = val8;
    pr.A = d.A;
    pr.nnz = (int32_t)d.nnz;
    pr.K = d.B * d.C * d.D;
    pr.CD = d.C * d.D;
    pr.D = d.D;
    pr.B = d.B;
    pr.stride = d.stride;
    pr.Ws = p.Ws;
    pr.rowb = p.rowb;
    pr.pixb = p.pixb;
    pr.divCD = make_fastdiv((uint32_t)pr.CD);
    pr.divD = make_fastdiv((uint32_t)d.D);
    pr.divS = make_fastdiv((uint32_t)d.stride);
    pr.divPG = make_fastdiv((uint32_t)(d.A / d.groups));
    hipLaunchKernelGGL(k_csr_prep, dim3((d.A + 3) / 4), dim3(256), 0, stream, pr);
    return check_hip(hipGetLastError(), "k_csr_prep");
}

int sp_launch(const sa_sparse_conv_desc &d, const SpPlan &p, const int32_t *rowp8, const int32_t *off8,
              const uint16_t *val8, hipStream_t stream) {
    SpConvArgs a;
    a.X = d.X;
    a.Y = d.Y;
    a.rowp8 = rowp8;
    a.off8 = off8;
    a.val8 = val8;
    a.x_bytes = (uint32_t)((int64_t)d.N * d.H * d.W * d.Cx * 2);
    a.N = d.N;
    a.H = d.H;
    a.W = d.W;
    a.Cx = d.Cx;
    a.A = d.A;
    a.B = d.B;
    a.C = d.C;
    a.stride = d.stride;
    a.pad = d.pad;
    a.P = p.P;
    a.Q = p.Q;
    a.NPQ = p.NPQ;
    a.Hp = p.Hp;
    a.Wp = p.Wp;
    a.Ws = p.Ws;
    a.Wpp = p.Wpp;
    a.rowb = p.rowb;
    a.nch = p.nch;
    a.pixb = p.pixb;
    a.per_group = d.A / d.groups;
    const int fbs = p.RPW * p.NW;  // filters per workgroup
    a.fb_per_group = (a.per_group + fbs - 1) / fbs;
    a.nfb = a.fb_per_group * d.groups;
    const int64_t ntiles = (p.NPQ + 64 * p.TN - 1) / (64 * p.TN);
    if (ntiles * a.nfb >= (int64_t(1) << 31)) return fail(SA_E_UNSUPPORTED, "conv_sparse: grid too large");
    a.nblocks = (int)(ntiles * a.nfb);
    a.divQ = make_fastdiv((uint32_t)p.Q);
    a.divP = make_fastdiv((uint32_t)p.P);
    a.divHp = make_fastdiv((uint32_t)p.Hp);
    a.divS = make_fastdiv((uint32_t)d.stride);
    a.divFbg = make_fastdiv((uint32_t)a.fb_per_group);
    a.divNch = make_fastdiv((uint32_t)p.nch);
    a.divRowc = make_fastdiv((uint32_t)(p.Wp * p.nch));
    if (p.RPW == 1)
        return p.NW == 16 ? launch_conv_csr<1, 16, 1>(a, p.lds, stream) : launch_conv_csr<1, 8, 1>(a, p.lds, stream);
    if (p.NW == 16)
        return p.TN == 2 ? launch_conv_csr<2, 16, 8>(a, p.lds, stream) : launch_conv_csr<1, 16, 8>(a, p.lds, stream);
    return p.TN == 2 ? launch_conv_csr<2, 8, 8>(a, p.lds, stream) : launch_conv_csr<1, 8, 8>(a, p.lds, stream);
}

}  // namespace
}  // namespace sa

using namespace sa;

extern "C" int structadmm_csr(const sa_csr_desc *desc, hipStream_t stream) {
    clear_error();
    if (!desc) return fail(SA_E_ARG, "csr: desc is required");
    const sa_csr_desc &d = *desc;
    if (d.A <= 0 || d.B <= 0 || d.C <= 0 || d.D <= 0)
        return fail(SA_E_ARG, "csr: A, B, C, D must be positive");
    const int64_t K = d.B * d.C * d.D, n = d.A * K;
    if (K >= (int64_t(1) << 31) || n >= (int64_t(1) << 31))
        return fail(SA_E_UNSUPPORTED, "csr: A*B*C*D must be below 2^31");
    if (d.nnz < 0 || d.nnz > n) return fail(SA_E_ARG, "csr: nnz=%lld outside [0, A*B*C*D]", (long long)d.nnz);
    if (!d.Z || !d.row_ptr) return fail(SA_E_ARG, "csr: Z and row_ptr are required");
    if (d.nnz > 0 && (!d.kept_idx || !d.col || !d.val))
        return fail(SA_E_ARG, "csr: kept_idx, col and val are required when nnz > 0");
    if (!aligned(d.Z, 4) || !aligned(d.row_ptr, 4) || (d.kept_idx && !aligned(d.kept_idx, 4)) ||
        (d.col && !aligned(d.col, 4)) || (d.val && !aligned(d.val, 2)))
        return fail(SA_E_ALIGN, "csr: arrays must be aligned to their element size");
    CsrArgs a;
    a.Z = d.Z;
    a.kept = d.kept_idx;
    a.row_ptr = d.row_ptr;
    a.col = d.col;
    a.val = d.val;
    a.A = (int32_t)d.A;
    a.K = (int32_t)K;
    a.nnz = (int32_t)d.nnz;
    a.n = (uint32_t)n;
    a.divK = make_fastdiv((uint32_t)K);
    const int blocks = (int)((d.nnz + 1 + 255) / 256);
    hipLaunchKernelGGL(k_csr_from_kept, dim3(blocks), dim3(256), 0, stream, a);
    return check_hip(hipGetLastError(), "k_csr_from_kept");
}

extern "C" size_t structadmm_conv_sparse_workspace(const sa_sparse_conv_desc *desc) {
    if (!desc) return 0;
    SpPlan p;
    if (sp_plan(*desc, &p) != SA_OK) {
        clear_error();
        return 0;
    }
    return p.ws_need;
}

extern "C" int structadmm_conv_sparse_fwd(const sa_sparse_conv_desc *desc, hipStream_t stream) {
    clear_error();
    if (!desc) return fail(SA_E_ARG, "conv_sparse: desc is required");
    const sa_sparse_conv_desc &d = *desc;
    SpPlan p;
    if (int rc = sp_plan(d, &p)) return rc;
    if (!d.X || !d.Y || !d.row_ptr) return fail(SA_E_ARG, "conv_sparse: X, Y and row_ptr are required");
    if (d.nnz > 0 && (!d.col || !d.val)) return fail(SA_E_ARG, "conv_sparse: col and val are required when nnz > 0");
    if (!aligned(d.X, 16) || !aligned(d.Y, 16) || !aligned(d.row_ptr, 4) || (d.col && !aligned(d.col, 4)) ||
        (d.val && !aligned(d.val, 2)))
        return fail(SA_E_ALIGN, "conv_sparse: X and Y must be 16-byte aligned, the CSR arrays to their element size");
    if (!d.ws || d.ws_bytes < p.ws_need)
        return fail(SA_E_WORKSPACE, "conv_sparse: scratch of %zu bytes required (%zu given)", p.ws_need,
                    d.ws ? d.ws_bytes : 0);
    if (!aligned(d.ws, 256)) return fail(SA_E_ALIGN, "conv_sparse: scratch must be 256-byte aligned");

    uint8_t *ws = static_cast<uint8_t *>(d.ws);
    int32_t *rowp8 = reinterpret_cast<int32_t *>(ws);
    int32_t *off8 = reinterpret_cast<int32_t *>(ws + p.off_at);
    uint16_t *val8 = reinterpret_cast<uint16_t *>(ws + p.val_at);

    if (!d.reuse_ws) {
        if (int rc = sp_prepare(d, p, rowp8, off8, val8, stream)) return rc;
    }
    return sp_launch(d, p, rowp8, off8, val8, stream);
}
