// gfx950 kernels and entry points that lay data out for the compacted CONV:
//   structadmm_compact    the dense GEMM matrix left after row (filter) and
//                         column (channel / filter-shape) pruning (Section 3,
//                         "Combination of structured sparsities"), in bfloat16
//   structadmm_pack_nhwc  binary32 NCHW activations -> bfloat16 NHWC, with an
//                         optional channel gather (the input a compacted
//                         predecessor layer would emit)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstring>
#include <vector>

#include "sa_device.h"
#include "sa_host.h"
#include "structadmm.h"

namespace sa {
namespace {

constexpr int kCompThreads = 1024;
constexpr int kCS = 8;  // ints per conv group in the size record

struct CompArgs {
    const float *Z;
    const uint8_t *row_mask, *col_mask, *chan_mask, *in_ch_mask;
    uint16_t *Wc;
    int32_t *row_idx, *col_ch, *col_tap;
    int32_t *counts;  // ws: [groups][kCS] = M, K, run, run_base, ch_lo, ch_span, kpad, run offset in the window
    int32_t A, B, C, D, groups, in_compacted;
};

// Is column candidate (tap t, channel b) of conv group gc kept?
__device__ inline bool col_kept(const CompArgs &a, int gc, int t, int b) {
    const int taps = a.C * a.D;
    if (a.col_mask && !a.col_mask[b * taps + t]) return false;
    if (a.chan_mask && !a.chan_mask[b]) return false;
    if (a.in_ch_mask && !a.in_ch_mask[gc * a.B + b]) return false;
    return true;
}

// Input-channel position of full channel `full` (compacted input: rank among set in_ch_mask).
__device__ inline int in_position(const CompArgs &a, int full) {
    if (!a.in_compacted) return full;
    int pos = 0;
    for (int q = 0; q < full; ++q) pos += a.in_ch_mask[q] != 0;
    return pos;
}

// Per conv group: M (kept rows), K (kept columns), the span of input channels
// the kept columns read and, when every tap keeps the same channels and their
// input positions are consecutive, that channel run -- for a channel-compacted
// input of a multiple of 8 channels widened to its enclosing 8-aligned window
// of positions when that is at most 1.5 times the run (the added positions
// become +0 columns).
__global__ __launch_bounds__(kCompThreads) void k_compact_count(CompArgs a) {
    __shared__ uint32_t tmp[kCompThreads / kWave + 1];
    __shared__ int s_first, s_last, s_cfirst, s_clast;
    const int gc = blockIdx.x;
    const int Ag = a.A / a.groups, taps = a.C * a.D;
    if (threadIdx.x == 0) {
        s_first = -1;
        s_last = -1;
        s_cfirst = -1;
        s_clast = -1;
    }
    __syncthreads();
    uint32_t m = 0, kc = 0, nb = 0;
    for (int r = threadIdx.x; r < Ag; r += kCompThreads) m += (!a.row_mask || a.row_mask[gc * Ag + r]) ? 1 : 0;
    // first and last kept channel: per thread, then per wavefront, then one
    // LDS atomic per wavefront (a dense layer keeps every candidate)
    int cf = INT_MAX, cl = -1;
    for (int64_t i = threadIdx.x; i < (int64_t)taps * a.B; i += kCompThreads) {
        int t = (int)(i / a.B), b = (int)(i - (int64_t)t * a.B);
        if (col_kept(a, gc, t, b)) {
            ++kc;
            cf = min(cf, b);
            cl = max(cl, b);
        }
    }
    // kept channels ignoring the shape mask (defines the run when there is no shape mask)
    int bf = INT_MAX, bl = -1;
    for (int b = threadIdx.x; b < a.B; b += kCompThreads) {
        bool keep = (!a.chan_mask || a.chan_mask[b]) && (!a.in_ch_mask || a.in_ch_mask[gc * a.B + b]);
        nb += keep ? 1 : 0;
        if (keep) {
            bf = min(bf, b);
            bl = max(bl, b);
        }
    }
    cf = wave_min_i32(cf);
    cl = wave_max_i32(cl);
    bf = wave_min_i32(bf);
    bl = wave_max_i32(bl);
    if ((threadIdx.x & (kWave - 1)) == 0) {
        if (cl >= 0) {
            atomicMin(reinterpret_cast<unsigned *>(&s_cfirst), (unsigned)cf);  // -1 is the largest unsigned
            atomicMax(&s_clast, cl);
        }
        if (bl >= 0) {
            atomicMin(reinterpret_cast<unsigned *>(&s_first), (unsigned)bf);
            atomicMax(&s_last, bl);
        }
    }
    // channels of the compacted input (every set bit of in_ch_mask)
    uint32_t ncx_part = 0;
    if (a.in_compacted)
        for (int c = threadIdx.x; c < a.groups * a.B; c += kCompThreads) ncx_part += a.in_ch_mask[c] != 0;
    uint32_t tot_m, tot_k, tot_b, ncx;
    block_excl_scan(m, tmp, &tot_m);
    block_excl_scan(kc, tmp, &tot_k);
    block_excl_scan(nb, tmp, &tot_b);
    block_excl_scan(ncx_part, tmp, &ncx);
    if (threadIdx.x == 0) {
        int run = 0, base = 0, kpad = 0, roff = 0;
        if (!a.col_mask && tot_b > 0) {
            int p0 = in_position(a, gc * a.B + s_first);
            int p1 = in_position(a, gc * a.B + s_last);
            if (p1 - p0 + 1 == (int)tot_b) {
                run = (int)tot_b;
                base = p0;
            }
        }
        int clo = 0, cspan = 0;
        if (tot_k > 0) {
            clo = in_position(a, gc * a.B + s_cfirst);
            cspan = in_position(a, gc * a.B + s_clast) - clo + 1;
        }
        if (run > 0 && a.in_compacted && ((base | run) & 7)) {
            const int lo = base & ~7, hi = (base + run + 7) & ~7;
            if ((ncx & 7) == 0 && hi <= (int)ncx && 2 * (hi - lo) <= 3 * run) {
                kpad = (hi - lo - run) * taps;
                roff = base - lo;
                tot_k += (uint32_t)kpad;
                run = hi - lo;
                base = lo;
                clo = lo;
                cspan = hi - lo;
            }
        }
        a.counts[kCS * gc + 0] = (int)tot_m;
        a.counts[kCS * gc + 1] = (int)tot_k;
        a.counts[kCS * gc + 2] = run;
        a.counts[kCS * gc + 3] = base;
        a.counts[kCS * gc + 4] = clo;
        a.counts[kCS * gc + 5] = cspan;
        a.counts[kCS * gc + 6] = kpad;
        a.counts[kCS * gc + 7] = roff;
    }
}

// Column-table entry of an alignment column: input position p, encoded
// below zero until k_compact_inpos (which maps kept channels to positions).
__device__ inline int32_t pad_code(int p) { return -p - 1; }

// Column tables (full input channel for now) and kept rows, concatenated over groups.
__global__ __launch_bounds__(kCompThreads) void k_compact_tables(CompArgs a) {
    __shared__ uint32_t tmp[kCompThreads / kWave + 1];
    const int gc = blockIdx.x;
    const int Ag = a.A / a.groups, taps = a.C * a.D;
    int row_off = 0, col_off = 0;
    for (int g = 0; g < gc; ++g) {
        row_off += a.counts[kCS * g + 0];
        col_off += a.counts[kCS * g + 1];
    }
    // a dense channel run is listed tap-major (the direct CONV reads 8
    // consecutive channels of one tap per load); any other column set
    // channel-major, so that every channel range is one range of columns
    const bool tap_major = a.counts[kCS * gc + 2] > 0;
    // a widened run: kept channel r of tap t goes to column t * run + roff + r,
    // the window's other positions to +0 alignment columns
    const int kpad = a.counts[kCS * gc + 6];
    const int wrun = a.counts[kCS * gc + 2], roff = a.counts[kCS * gc + 7];
    const int krun = kpad > 0 ? wrun - kpad / taps : 0;  // kept channels per tap
    if (kpad > 0) {
        const int wbase = a.counts[kCS * gc + 3];
        for (int idx = threadIdx.x; idx < taps * wrun; idx += kCompThreads) {
            const int t = idx / wrun, q = idx - t * wrun;
            if (q < roff || q >= roff + krun) {
                a.col_ch[col_off + idx] = pad_code(wbase + q);
                a.col_tap[col_off + idx] = t;
            }
        }
    }
    uint32_t running = 0;
    const int64_t ncand = (int64_t)taps * a.B;
    for (int64_t base = 0; base < ncand; base += kCompThreads) {
        int64_t i = base + threadIdx.x;
        bool keep = false;
        int t = 0, b = 0;
        if (i < ncand) {
            if (tap_major) {
                t = (int)(i / a.B);
                b = (int)(i - (int64_t)t * a.B);
            } else {
                b = (int)(i / taps);
                t = (int)(i - (int64_t)b * taps);
            }
            keep = col_kept(a, gc, t, b);
        }
        uint32_t tot;
        uint32_t pos = running + block_excl_scan(keep ? 1u : 0u, tmp, &tot);
        if (keep) {
            // tap-major with every tap keeping the same channels: pos = t * krun + rank
            const int j = kpad > 0 ? t * wrun + roff + ((int)pos - t * krun) : (int)pos;
            a.col_ch[col_off + j] = gc * a.B + b;
            a.col_tap[col_off + j] = t;
        }
        running += tot;
    }
    running = 0;
    for (int base = 0; base < Ag; base += kCompThreads) {
        int r = base + threadIdx.x;
        bool keep = r < Ag && (!a.row_mask || a.row_mask[gc * Ag + r]);
        uint32_t tot;
        uint32_t pos = running + block_excl_scan(keep ? 1u : 0u, tmp, &tot);
        if (keep) a.row_idx[row_off + pos] = gc * Ag + r;
        running += tot;
    }
}

// Wc rows: block (m, gc) writes row m of group gc: bf16(Z[a, b, c, d]) per column, 0 padding.
__global__ __launch_bounds__(256) void k_compact_gather(CompArgs a) {
    const int m = blockIdx.x, gc = blockIdx.y;
    const int M = a.counts[kCS * gc + 0];
    if (m >= M) return;
    const int K = a.counts[kCS * gc + 1];
    const int ldk = (K + 63) / 64 * 64;
    int64_t wc_off = 0;
    int row_off = 0, col_off = 0;
    for (int g = 0; g < gc; ++g) {
        const int Mg = a.counts[kCS * g + 0], Kg = a.counts[kCS * g + 1];
        wc_off += (int64_t)Mg * ((Kg + 63) / 64 * 64);
        row_off += Mg;
        col_off += Kg;
    }
    const int row = a.row_idx[row_off + m];
    uint16_t *dst = a.Wc + wc_off + (int64_t)m * ldk;
    for (int j = threadIdx.x; j < ldk; j += blockDim.x) {
        uint16_t v = 0;
        if (j < K && a.col_ch[col_off + j] >= 0) {  // alignment columns hold +0
            const int b = a.col_ch[col_off + j] - gc * a.B;
            const int t = a.col_tap[col_off + j];
            const int c = t / a.D, d = t - (t / a.D) * a.D;
            v = f32_to_bf16_bits(a.Z[(((int64_t)row * a.B + b) * a.C + c) * a.D + d]);
        }
        dst[j] = v;
    }
}

// Full input channel -> position in the channel-compacted input.
__global__ __launch_bounds__(kCompThreads) void k_compact_inpos(CompArgs a, int total_cols) {
    extern __shared__ int32_t pos[];  // [groups*B]
    __shared__ uint32_t tmp[kCompThreads / kWave + 1];
    const int nch = a.groups * a.B;
    uint32_t running = 0;
    for (int base = 0; base < nch; base += kCompThreads) {
        int c = base + threadIdx.x;
        uint32_t f = (c < nch && a.in_ch_mask[c]) ? 1u : 0u;
        uint32_t tot;
        uint32_t p = running + block_excl_scan(f, tmp, &tot);
        if (c < nch) pos[c] = (int32_t)p;
        running += tot;
    }
    __syncthreads();
    for (int j = threadIdx.x; j < total_cols; j += kCompThreads) {
        const int full = a.col_ch[j];
        a.col_ch[j] = full < 0 ? -full - 1 : (full < nch ? pos[full] : 0);  // alignment columns: their position
    }
}

// ---------------------------------------------------------------- pack
constexpr int kPackTile = 64;

// X binary32 NCHW -> Xp bfloat16 NHWC with kept channels in ascending order.
// Workgroup = 64 channels x 64 pixels of one image: float4 loads along the
// pixels, bf16 conversion, transpose through LDS with every kept channel at
// its output rank, 16-byte stores along the channels when aligned.
__global__ __launch_bounds__(256) void k_pack_nhwc(const float *__restrict__ X, const uint8_t *__restrict__ keep,
                                                   uint16_t *__restrict__ Xp, int Cin, int HW, int Cx) {
    __shared__ __attribute__((aligned(16))) uint16_t tile[kPackTile][kPackTile + 8];  // [pixel][rank]
    __shared__ int32_t crank[kPackTile];
    __shared__ int32_t s_base, s_nkept;
    const int p0 = blockIdx.x * kPackTile, c0 = blockIdx.y * kPackTile, n = blockIdx.z;
    const int tid = threadIdx.x;
    if (tid < kWave) {
        // rank of channel c0 among the kept channels, then ranks inside the tile
        uint32_t cnt = 0;
        if (keep)
            for (int c = tid; c < c0; c += kWave) cnt += keep[c] != 0;
        else
            cnt = (tid == 0) ? (uint32_t)c0 : 0u;
        cnt = wave_sum_u32(cnt);
        const int c = c0 + tid;
        const uint32_t f = (c < Cin && (!keep || keep[c])) ? 1u : 0u;
        const uint32_t incl = wave_incl_scan(f);
        crank[tid] = f ? (int32_t)(incl - 1) : -1;
        if (tid == 0) s_base = (int32_t)cnt;
        if (tid == kWave - 1) s_nkept = (int32_t)incl;
    }
    __syncthreads();
    const int nk = s_nkept, base = s_base;
    if (nk == 0) return;
    const bool vec_in = (HW % 4) == 0;
    for (int i = tid; i < kPackTile * (kPackTile / 4); i += 256) {
        const int cl = i / (kPackTile / 4), pq = i % (kPackTile / 4);
        const int r = crank[cl];
        if (r < 0) continue;
        const int p = p0 + pq * 4;
        const float *src = X + ((int64_t)n * Cin + c0 + cl) * HW + p;
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        if (vec_in && p + 4 <= HW) {
            const float4 t = *reinterpret_cast<const float4 *>(src);
            v[0] = t.x;
            v[1] = t.y;
            v[2] = t.z;
            v[3] = t.w;
        } else {
            for (int e = 0; e < 4; ++e)
                if (p + e < HW) v[e] = src[e];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) tile[pq * 4 + e][r] = f32_to_bf16_bits(v[e]);
    }
    __syncthreads();
    if ((Cx % 8) == 0 && (base % 8) == 0) {
        const int chunks = (nk + 7) / 8;
        for (int i = tid; i < kPackTile * chunks; i += 256) {
            const int pl = i / chunks, ch = i % chunks;
            const int p = p0 + pl;
            if (p >= HW) continue;
            uint16_t *dst = Xp + ((int64_t)n * HW + p) * Cx + base;
            if (ch * 8 + 8 <= nk && base + ch * 8 + 8 <= Cx) {
                *reinterpret_cast<uint4 *>(dst + ch * 8) = *reinterpret_cast<const uint4 *>(&tile[pl][ch * 8]);
            } else {
                for (int e = ch * 8; e < nk && e < ch * 8 + 8; ++e)
                    if (base + e < Cx) dst[e] = tile[pl][e];
            }
        }
    } else {
        for (int i = tid; i < kPackTile * nk; i += 256) {
            const int pl = i / nk, e = i % nk;
            const int p = p0 + pl;
            if (p < HW && base + e < Cx) Xp[((int64_t)n * HW + p) * Cx + base + e] = tile[pl][e];
        }
    }
}

// Few input channels and no channel gather: one thread per pixel.
__global__ __launch_bounds__(256) void k_pack_small(const float *__restrict__ X, uint16_t *__restrict__ Xp, int Cin,
                                                    int HW, int64_t pixels) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < pixels; i += (int64_t)gridDim.x * 256) {
        const int64_t n = i / HW, p = i - n * HW;
        for (int c = 0; c < Cin; ++c) Xp[i * Cin + c] = f32_to_bf16_bits(X[(n * Cin + c) * HW + p]);
    }
}

}  // namespace
}  // namespace sa

using namespace sa;

namespace {

int check_compact(const sa_compact_desc &d) {
    if (int rc = validate_compact(d)) return rc;
    if (d.in_compacted && (int64_t)d.groups * d.B > 16384)
        return fail(SA_E_UNSUPPORTED, "compact: in_compacted supports at most 16384 input channels");
    return SA_OK;
}

CompArgs compact_args(const sa_compact_desc &d) {
    CompArgs a;
    memset(&a, 0, sizeof a);
    a.Z = d.Z;
    a.row_mask = d.row_mask;
    a.col_mask = d.col_mask;
    a.chan_mask = d.chan_mask;
    a.in_ch_mask = d.in_ch_mask;
    a.Wc = d.Wc;
    a.row_idx = d.row_idx;
    a.col_ch = d.col_ch;
    a.col_tap = d.col_tap;
    a.counts = static_cast<int32_t *>(d.ws);
    a.A = (int)d.A;
    a.B = (int)d.B;
    a.C = (int)d.C;
    a.D = (int)d.D;
    a.groups = d.groups;
    a.in_compacted = d.in_compacted ? 1 : 0;
    return a;
}

// The kernels of one compaction that need no host decision: the per-group
// counts (into ws), the column tables and kept rows, the gathered matrix.
int launch_compact(const CompArgs &a, hipStream_t stream) {
    const int Ag = a.A / a.groups;
    hipLaunchKernelGGL(k_compact_count, dim3(a.groups), dim3(kCompThreads), 0, stream, a);
    if (int rc = check_hip(hipGetLastError(), "k_compact_count")) return rc;
    hipLaunchKernelGGL(k_compact_tables, dim3(a.groups), dim3(kCompThreads), 0, stream, a);
    if (int rc = check_hip(hipGetLastError(), "k_compact_tables")) return rc;
    hipLaunchKernelGGL(k_compact_gather, dim3(Ag, a.groups), dim3(256), 0, stream, a);
    return check_hip(hipGetLastError(), "k_compact_gather");
}

int total_columns(const int32_t *counts, int groups) {
    int total = 0;
    for (int g = 0; g < groups; ++g) total += counts[kCS * g + 1];
    return total;
}

// For a channel-compacted input: input positions in the column tables.
int launch_inpos(const CompArgs &a, const int32_t *counts, hipStream_t stream) {
    const int total = total_columns(counts, a.groups);
    if (!a.in_compacted || total == 0) return SA_OK;
    const size_t lds = sizeof(int32_t) * (size_t)a.groups * a.B;
    hipLaunchKernelGGL(k_compact_inpos, dim3(1), dim3(kCompThreads), lds, stream, a, total);
    return check_hip(hipGetLastError(), "k_compact_inpos");
}

void fill_sizes(const int32_t *counts, int groups, sa_compact_sizes *sizes) {
    memset(sizes, 0, sizeof *sizes);
    sizes->groups = groups;
    int64_t wc_off = 0;
    int32_t row_off = 0, col_off = 0;
    for (int g = 0; g < groups; ++g) {
        sizes->M[g] = counts[kCS * g + 0];
        sizes->K[g] = counts[kCS * g + 1];
        sizes->ldk[g] = (sizes->K[g] + 63) / 64 * 64;
        sizes->run[g] = counts[kCS * g + 2];
        sizes->run_base[g] = counts[kCS * g + 3];
        sizes->ch_lo[g] = counts[kCS * g + 4];
        sizes->ch_span[g] = counts[kCS * g + 5];
        sizes->kpad[g] = counts[kCS * g + 6];
        sizes->wc_offset[g] = wc_off;
        sizes->row_offset[g] = row_off;
        sizes->col_offset[g] = col_off;
        wc_off += (int64_t)sizes->M[g] * sizes->ldk[g];
        row_off += sizes->M[g];
        col_off += sizes->K[g];
    }
}

}  // namespace

extern "C" int structadmm_compact(const sa_compact_desc *desc, sa_compact_sizes *sizes, hipStream_t stream) {
    clear_error();
    if (!desc || !sizes) return fail(SA_E_ARG, "compact: desc and sizes are required");
    return structadmm_compact_many(desc, 1, sizes, stream);
}

extern "C" int structadmm_compact_many(const sa_compact_desc *descs, int32_t n, sa_compact_sizes *sizes,
                                       hipStream_t stream) {
    clear_error();
    if (n < 0 || (n > 0 && (!descs || !sizes))) return fail(SA_E_ARG, "compact: descs and sizes are required");
    // every descriptor is checked before anything is enqueued
    for (int i = 0; i < n; ++i) {
        if (int rc = check_compact(descs[i])) return rc;
        const uintptr_t wi = reinterpret_cast<uintptr_t>(descs[i].ws);
        for (int j = 0; j < i; ++j) {
            const uintptr_t wj = reinterpret_cast<uintptr_t>(descs[j].ws);
            if (wi < wj + SA_COMPACT_WS_BYTES && wj < wi + SA_COMPACT_WS_BYTES)
                return fail(SA_E_ARG, "compact: descriptors %d and %d share scratch", j, i);
        }
    }
    if (n == 0) return SA_OK;
    std::vector<CompArgs> args(n);
    for (int i = 0; i < n; ++i) {
        args[i] = compact_args(descs[i]);
        if (int rc = launch_compact(args[i], stream)) return rc;
    }
    std::vector<int32_t> counts((size_t)n * kCS * SA_MAX_CONV_GROUPS);
    for (int i = 0; i < n; ++i)
        if (int rc = check_hip(hipMemcpyAsync(&counts[(size_t)i * kCS * SA_MAX_CONV_GROUPS], descs[i].ws,
                                              sizeof(int32_t) * kCS * descs[i].groups, hipMemcpyDeviceToHost, stream),
                               "compact: copy sizes"))
            return rc;
    if (int rc = check_hip(hipStreamSynchronize(stream), "compact: synchronize")) return rc;
    bool inpos = false;
    for (int i = 0; i < n; ++i) {
        const int32_t *c = &counts[(size_t)i * kCS * SA_MAX_CONV_GROUPS];
        if (args[i].in_compacted && total_columns(c, args[i].groups) > 0) {
            if (int rc = launch_inpos(args[i], c, stream)) return rc;
            inpos = true;
        }
    }
    if (inpos)
        if (int rc = check_hip(hipStreamSynchronize(stream), "compact: synchronize")) return rc;
    for (int i = 0; i < n; ++i) fill_sizes(&counts[(size_t)i * kCS * SA_MAX_CONV_GROUPS], args[i].groups, &sizes[i]);
    return SA_OK;
}

extern "C" int structadmm_pack_nhwc(const float *X, int32_t N, int32_t Cin, int32_t H, int32_t W,
                                    const uint8_t *keep, int32_t Cx, uint16_t *Xp, hipStream_t stream) {
    clear_error();
    if (!X || !Xp) return fail(SA_E_ARG, "pack: X and Xp are required");
    if (N <= 0 || Cin <= 0 || H <= 0 || W <= 0 || Cx <= 0 || Cx > Cin)
        return fail(SA_E_ARG, "pack: sizes must be positive and Cx <= Cin");
    if (!keep && Cx != Cin) return fail(SA_E_ARG, "pack: Cx must equal Cin without a keep mask");
    if ((int64_t)H * W > (int64_t(1) << 30) || (int64_t)Cin > 65535 || (int64_t)N > 65535)
        return fail(SA_E_UNSUPPORTED, "pack: tensor too large");
    const int HW = H * W;
    if (!keep && Cin <= 8) {
        const int64_t pixels = (int64_t)N * HW;
        const int blocks = (int)std::min<int64_t>(8192, (pixels + 255) / 256);
        hipLaunchKernelGGL(k_pack_small, dim3(blocks), dim3(256), 0, stream, X, Xp, Cin, HW, pixels);
        return check_hip(hipGetLastError(), "k_pack_small");
    }
    dim3 grid((HW + kPackTile - 1) / kPackTile, (Cin + kPackTile - 1) / kPackTile, N);
    hipLaunchKernelGGL(k_pack_nhwc, grid, dim3(256), 0, stream, X, keep, Xp, Cin, HW, Cx);
    return check_hip(hipGetLastError(), "k_pack_nhwc");
}
