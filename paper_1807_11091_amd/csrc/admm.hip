// gfx950 kernels and entry points of the ADMM Z-update (projection onto the
// sparsity sets of Section 3, as solved in Section 4), of the dual update /
// gradient of eq. (3), and of the W-subproblem's SGD step, also used for masked
// retraining (k_sgd).
//
// Data flow of structadmm_project for one dependency level of layers:
//   k_expand_allowed  (channel, shape and element-wise layers with an input-channel
//                     support) per-column support bytes; filter sets read the mask
//   k_row_scores      filter sets: one wavefront per weight row, O_a in binary64
//   k_col_partials    channel / shape sets: binary64 column sums per band of rows
//   k_select          one workgroup per structured layer: final scores, radix
//                     select of the k-th largest score bits in LDS, lowest-index
//                     tie-break, mask + ascending kept_idx, per-column keep bytes
//   k_elem_*          non-structured sets: 3 histogram passes over |v| bits, then an
//                     order-preserving count / scan / apply
//   k_apply           flat streaming Z (+ fused U', G) writer over every layer
// Every reduction has a fixed order; no floating-point atomics are used.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <vector>

#include "sa_device.h"
#include "sa_host.h"
#include "structadmm.h"

namespace sa {
namespace {

constexpr int kTab = 64;           // layers per launch (kernel-argument table, < 8 KiB; ResNet-50's
                                   // 53 convolutions take one launch per phase)
constexpr int kRowThreads = 256;   // 4 wavefronts, one weight row each at a time
constexpr int kRowItems = 2;       // work items per wavefront
constexpr int kColThreads = 256;
constexpr int kColBand = 32;       // rows per band of column partial sums
constexpr int kColSlices = 4;      // row slices of a band (one wavefront each)
constexpr int kSelThreads = 1024;
constexpr int kElemThreads = 256;
constexpr int kElemPerThread = 8;
constexpr int kElemChunk = kElemThreads * kElemPerThread;  // elements per workgroup
constexpr int kElemHistBlocks = 1024;

// ---------------------------------------------------------------- tables
struct RowLayer {
    const float *W;
    float *U;
    const uint8_t *allowed;  // [groups*K] or null: every entry inside the support
    const uint8_t *inmask;   // [groups*B] or null: filter sets read the support from the
                             // input-channel mask itself (entry (a, j) is inside when
                             // inmask[(a / Ag) * B + j / CD] is set)
    double *scores;          // [A] (row scores)
    double *rowpart;         // [A][nchunk] partial row sums when nchunk > 1
    int32_t A, K, Ag;        // rows, row length, rows per conv group
    int32_t R, nchunk;       // rows per wavefront item (short rows), 1024-weight chunks per row
    int32_t vec;             // K % 4 == 0: float4 path
    int32_t B;               // input channels per conv group (inmask)
    FastDiv divCD;           // taps per channel (inmask)
    float rho;
};
struct RowTab {
    RowLayer L[kTab];
    int32_t begin[kTab + 1];
    int32_t nl;
};

struct ColLayer {
    const float *W;
    const float *U;
    const uint8_t *allowed;
    double *partials;  // [nbands][K]
    int32_t A, K, Ag, nbands, ctiles, vec;
};
struct ColTab {
    ColLayer L[kTab];
    int32_t begin[kTab + 1];
    int32_t nl;
};

struct SelLayer {
    const double *partials;  // channel / shape: [nbands][K]
    const double *rowpart;   // filter with chunked rows: [G][nchunk]
    double *scores;          // [G]: filter: input (or output with rowpart); channel / shape: output
    uint8_t *mask;           // [G]
    int32_t *kept_idx;       // [k]
    uint8_t *colkeep;        // [groups*K] or null
    const uint8_t *allowed;  // [groups*K] or null
    int32_t kind, G, k, K, CD, nbands, groups, nchunk;
};
struct SelTab {
    SelLayer L[kTab];
    int32_t nl;
};

struct DualLayer {
    const float *W;
    const float *Z;
    float *U;
    float *G;
    int32_t n, update;
    float rho;
};
struct DualTab {
    DualLayer L[kTab];
    int32_t begin[kTab + 1];
    int32_t nl;
};

struct SgdLayer {
    float *W;
    const float *Gf;
    const float *Z;
    const float *U;
    const uint8_t *mask;
    int32_t n, kind;
    FastDiv divK, divCD;  // entry -> filter, column -> channel
    float rho, lr;
};
struct SgdTab {
    SgdLayer L[kTab];
    int32_t begin[kTab + 1];
    int32_t nl;
};

__device__ inline int find_layer(const int32_t *begin, int nl, int b) {
    // the last layer whose first block is at or below b (binary search: a
    // launch holds up to 64 layers)
    int lo = 0, hi = nl - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (begin[mid] <= b) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Stores 4 consecutive binary32 values (16-byte aligned) with the
// non-temporal hint: streamed output that nothing reads back soon.
typedef float f32x4v __attribute__((ext_vector_type(4)));
__device__ inline void nt_store4(float *p, const float *v) {
    __builtin_nontemporal_store(f32x4v{v[0], v[1], v[2], v[3]}, reinterpret_cast<f32x4v *>(p));
}

// ---------------------------------------------------------------- support
// allowed[gc*K + j] = in_ch_mask[gc*B + j / CD]
__global__ void k_expand_allowed(const uint8_t *__restrict__ in_ch_mask, uint8_t *__restrict__ allowed,
                                 int groups, int B, int CD, int K) {
    int64_t total = (int64_t)groups * K;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        int gc = (int)(i / K);
        int j = (int)(i - (int64_t)gc * K);
        allowed[i] = in_ch_mask[gc * B + j / CD] ? 1 : 0;
    }
}

// ---------------------------------------------------------------- scores
__device__ inline float masked(float v, uint8_t keep) { return keep ? v : 0.0f; }

// O_a = sum_j (double)v_aj^2 for each filter a (Section 4, filter-wise set).
// Every wavefront takes one item: R = 4 rows when a row has at most 64 float4
// (one per lane), 2 rows up to 128, else one 1024-weight chunk of a row, whose
// partial sums k_select adds in chunk order.
__device__ inline float4 row_v(const RowLayer &L, const uint8_t *al, const uint8_t *im, int64_t base, int i) {
    float4 x = *reinterpret_cast<const float4 *>(L.W + base + 4 * (int64_t)i);
    float4 y = *reinterpret_cast<const float4 *>(L.U + base + 4 * (int64_t)i);
    float4 v = make_float4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
    if (al) {
        uchar4 m = reinterpret_cast<const uchar4 *>(al)[i];
        v.x = masked(v.x, m.x); v.y = masked(v.y, m.y);
        v.z = masked(v.z, m.z); v.w = masked(v.w, m.w);
    } else if (im) {  // the input channel of column j is j / CD
        const uint32_t j = 4u * (uint32_t)i;
        v.x = masked(v.x, im[fdiv(j, L.divCD)]); v.y = masked(v.y, im[fdiv(j + 1, L.divCD)]);
        v.z = masked(v.z, im[fdiv(j + 2, L.divCD)]); v.w = masked(v.w, im[fdiv(j + 3, L.divCD)]);
    }
    return v;
}
__device__ inline const uint8_t *row_inmask(const RowLayer &L, int a) {
    return L.inmask ? L.inmask + (int64_t)(a / L.Ag) * L.B : nullptr;
}
__device__ inline double sq4(float4 v) {
    double acc = (double)v.x * (double)v.x;
    acc += (double)v.y * (double)v.y;
    acc += (double)v.z * (double)v.z;
    acc += (double)v.w * (double)v.w;
    return acc;
}

__global__ __launch_bounds__(kRowThreads) void k_row_scores(RowTab tab) {
    const int li = find_layer(tab.begin, tab.nl, blockIdx.x);
    const RowLayer &L = tab.L[li];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    constexpr int kWaves = kRowThreads / kWave;
    // kRowItems consecutive work items per wavefront, all of their loads issued together
    const int item0 = ((blockIdx.x - tab.begin[li]) * kWaves + wave) * kRowItems;
    if (!L.vec) {  // item = row
        for (int a = item0; a < item0 + kRowItems && a < L.A; ++a) {
            const int64_t base = (int64_t)a * L.K;
            const uint8_t *al = L.allowed ? L.allowed + (int64_t)(a / L.Ag) * L.K : nullptr;
            const uint8_t *im = row_inmask(L, a);
            double acc = 0.0;
            for (int i = lane; i < L.K; i += kWave) {
                float v = L.W[base + i] + L.U[base + i];
                if (al) v = masked(v, al[i]);
                else if (im) v = masked(v, im[fdiv((uint32_t)i, L.divCD)]);
                acc += (double)v * (double)v;
            }
            acc = wave_sum(acc);
            if (lane == 0) L.scores[a] = acc;
        }
        return;
    }
    const int K4 = L.K >> 2;
    float4 v[kRowItems][4];
    if (L.R > 1) {  // item = R short rows; slot u: row a0 + u / (4 / R), float4 lane + 64 * (u % (4 / R))
        const int R = L.R;
#pragma unroll
        for (int q = 0; q < kRowItems; ++q)
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int a = (item0 + q) * R + u / (4 / R), i = lane + kWave * (u % (4 / R));
                v[q][u] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (a < L.A && i < K4) {
                    const uint8_t *al = L.allowed ? L.allowed + (int64_t)(a / L.Ag) * L.K : nullptr;
                    v[q][u] = row_v(L, al, row_inmask(L, a), (int64_t)a * L.K, i);
                }
            }
#pragma unroll
        for (int q = 0; q < kRowItems; ++q) {
            const int a0 = (item0 + q) * R;
            if (a0 >= L.A) break;
            double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int u = 0; u < 4; ++u) acc[u / (4 / R)] += sq4(v[q][u]);
            for (int r = 0; r < R; ++r) {
                const double t = wave_sum(acc[r]);
                if (lane == 0 && a0 + r < L.A) L.scores[a0 + r] = t;
            }
        }
        return;
    }
    // item = (row, chunk of 256 float4): long rows spread over several wavefronts
#pragma unroll
    for (int q = 0; q < kRowItems; ++q) {
        const int item = item0 + q;
        const int a = item / L.nchunk, c = item - a * L.nchunk;
        const uint8_t *al = (L.allowed && a < L.A) ? L.allowed + (int64_t)(a / L.Ag) * L.K : nullptr;
        const uint8_t *im = a < L.A ? row_inmask(L, a) : nullptr;
        const int64_t base = (int64_t)a * L.K;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = c * 4 * kWave + u * kWave + lane;
            v[q][u] = (a < L.A && i < K4) ? row_v(L, al, im, base, i) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
#pragma unroll
    for (int q = 0; q < kRowItems; ++q) {
        const int item = item0 + q;
        const int a = item / L.nchunk, c = item - a * L.nchunk;
        if (a >= L.A) break;
        double acc = 0.0;
#pragma unroll
        for (int u = 0; u < 4; ++u) acc += sq4(v[q][u]);
        acc = wave_sum(acc);
        if (lane == 0) {
            if (L.nchunk == 1) L.scores[a] = acc;
            else L.rowpart[(int64_t)a * L.nchunk + c] = acc;
        }
    }
}

// partials[band][j] = sum over rows a of the band of (double)v_aj^2
// (column sums; channel and shape scores are finished in k_select).  The four
// wavefronts of a workgroup take 8-row slices of the 32-row band; the slice
// sums are added in slice order.
__global__ __launch_bounds__(kColThreads) void k_col_partials(ColTab tab) {
    constexpr int kLanes = kColThreads / kColSlices;
    __shared__ double red[kColSlices - 1][kLanes * 4];
    const int li = find_layer(tab.begin, tab.nl, blockIdx.x);
    const ColLayer &L = tab.L[li];
    const int lb = blockIdx.x - tab.begin[li];
    const int band = lb / L.ctiles, ct = lb - band * L.ctiles;
    const int lane = threadIdx.x % kLanes, slice = threadIdx.x / kLanes;
    const int a0 = min(L.A, band * kColBand + slice * (kColBand / kColSlices));
    const int a1 = min(L.A, a0 + kColBand / kColSlices);
    const int cw = L.vec ? 4 : 1;  // columns per lane
    const int j = (ct * kLanes + lane) * cw;
    double s[4] = {0.0, 0.0, 0.0, 0.0};
    if (j < L.K) {
        if (L.vec) {
            for (int a = a0; a < a1; ++a) {
                const int64_t off = (int64_t)a * L.K + j;
                float4 x = *reinterpret_cast<const float4 *>(L.W + off);
                float4 y = *reinterpret_cast<const float4 *>(L.U + off);
                float v0 = x.x + y.x, v1 = x.y + y.y, v2 = x.z + y.z, v3 = x.w + y.w;
                if (L.allowed) {
                    uchar4 m = *reinterpret_cast<const uchar4 *>(L.allowed + (int64_t)(a / L.Ag) * L.K + j);
                    v0 = masked(v0, m.x); v1 = masked(v1, m.y);
                    v2 = masked(v2, m.z); v3 = masked(v3, m.w);
                }
                s[0] += (double)v0 * (double)v0;
                s[1] += (double)v1 * (double)v1;
                s[2] += (double)v2 * (double)v2;
                s[3] += (double)v3 * (double)v3;
            }
        } else {
            for (int a = a0; a < a1; ++a) {
                const int64_t off = (int64_t)a * L.K + j;
                float v = L.W[off] + L.U[off];
                if (L.allowed) v = masked(v, L.allowed[(int64_t)(a / L.Ag) * L.K + j]);
                s[0] += (double)v * (double)v;
            }
        }
    }
    if (slice > 0)
        for (int c = 0; c < 4; ++c) red[slice - 1][lane * 4 + c] = s[c];
    __syncthreads();
    if (slice == 0 && j < L.K) {
        double *p = L.partials + (int64_t)band * L.K + j;
        for (int c = 0; c < cw; ++c) {
            double t = s[c];
#pragma unroll
            for (int q = 0; q < kColSlices - 1; ++q) t += red[q][lane * 4 + c];
            p[c] = t;
        }
    }
}

// ---------------------------------------------------------------- select
// One workgroup per structured layer.  Keeps exactly k groups: the first k
// of the order (score descending, index ascending), i.e. every group whose
// score exceeds the k-th largest score T plus the lowest-index groups that
// tie with it.  Scores are non-negative binary64, so their bit patterns order
// like unsigned integers: T is found by an MSB-first radix select over the
// 64-bit keys (eight 8-bit digits, one LDS histogram per digit), and the ties
// are ranked by an ordered scan in index order.  Counting is order-free and
// the scans have a fixed order, so the result is reproducible.
__global__ __launch_bounds__(kSelThreads) void k_select(SelTab tab) {
    __shared__ uint64_t skey[SA_MAX_STRUCT_GROUPS];
    __shared__ uint8_t smask[SA_MAX_STRUCT_GROUPS];
    __shared__ uint32_t hist[256];
    __shared__ uint32_t scan_tmp[kSelThreads / kWave + 1];
    __shared__ uint64_t s_prefix;
    __shared__ uint32_t s_need, s_class;

    const SelLayer &L = tab.L[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63;
    const int G = L.G;

    // 1. final scores
    for (int g = tid; g < G; g += kSelThreads) {
        double s;
        if (L.kind == SA_FILTER) {
            if (L.rowpart) {  // chunk partials, added in chunk order
                s = 0.0;
                for (int c = 0; c < L.nchunk; ++c) s += L.rowpart[(int64_t)g * L.nchunk + c];
            } else {
                s = L.scores[g];
            }
        } else {
            // shape: over bands; channel: over taps, then bands.  The terms are
            // loaded 16 at a time (every load in flight together) and added in
            // that order; the padding terms past the end add +0 to a sum of
            // squares, which leaves it unchanged.
            const int taps = L.kind == SA_SHAPE ? 1 : L.CD, nb = L.nbands;
            const double *base = L.partials + (L.kind == SA_SHAPE ? g : g * L.CD);
            const int n = taps * nb;
            int t = 0, b = 0;
            s = 0.0;
            for (int i0 = 0; i0 < n; i0 += 16) {
                double v[16];
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    v[q] = i0 + q < n ? base[(int64_t)b * L.K + t] : 0.0;
                    if (++b == nb) {
                        b = 0;
                        ++t;
                    }
                }
#pragma unroll
                for (int q = 0; q < 16; ++q) s += v[q];
            }
        }
        if (L.kind != SA_FILTER || L.rowpart) L.scores[g] = s;
        skey[g] = (uint64_t)__double_as_longlong(s);
        smask[g] = 0;
    }
    __syncthreads();

    // 2. k-th largest key T, and how many of the keys equal to T are kept
    const int per = (G + kSelThreads - 1) / kSelThreads;
    const int g0 = min(G, tid * per), g1 = min(G, g0 + per);
    if (L.k > 0 && L.k < G) {
        uint64_t prefix = 0, pmask = 0;
        uint32_t need = (uint32_t)L.k;  // rank of T among the keys matching prefix
        for (int shift = 56; shift >= 0; shift -= 8) {
            if (tid < 256) hist[tid] = 0;
            __syncthreads();
            // the keys of a wavefront that share the first matching key's
            // digit are counted with one atomic (in the leading digits most
            // keys share one bin)
            for (int g0w = tid - lane; g0w < G; g0w += kSelThreads) {
                const int g = g0w + lane;
                const uint64_t key = g < G ? skey[g] : 0;
                const bool in = g < G && (key & pmask) == prefix;
                const uint32_t dig = (uint32_t)(key >> shift) & 255u;
                const unsigned long long vm = __ballot(in);
                if (vm) {
                    const int leader = (int)__builtin_ctzll(vm);
                    const uint32_t d0 = (uint32_t)__shfl((int)dig, leader);
                    const unsigned long long same = __ballot(in && dig == d0);
                    if (lane == leader) atomicAdd(&hist[d0], (uint32_t)__popcll(same));
                    if (in && dig != d0) atomicAdd(&hist[dig], 1u);
                }
            }
            __syncthreads();
            if (tid < kWave) {
                // lane l owns digits 255-4l .. 252-4l (descending)
                uint32_t c[4], tot = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) tot += (c[q] = hist[255 - 4 * lane - q]);
                const uint32_t incl = wave_incl_scan(tot), excl = incl - tot;
                if (excl < need && need <= incl) {
                    uint32_t cum = excl;
                    for (int q = 0; q < 4; ++q) {
                        if (cum + c[q] >= need) {
                            s_prefix = prefix | ((uint64_t)(255 - 4 * lane - q) << shift);
                            s_need = need - cum;
                            s_class = c[q];
                            break;
                        }
                        cum += c[q];
                    }
                }
            }
            __syncthreads();
            prefix = s_prefix;
            need = s_need;
            pmask |= (uint64_t)255 << shift;
            // every key of the class is kept: no finer digit matters (s_* are
            // rewritten only after the next pass's two barriers)
            if (s_class == need) break;
        }
        // keys whose leading digits exceed the class are kept; keys of the class
        // (all equal when every digit was resolved) are kept in index order
        uint32_t ties = 0;
        for (int g = g0; g < g1; ++g) ties += (skey[g] & pmask) == prefix;
        uint32_t total;
        uint32_t rank = block_excl_scan(ties, scan_tmp, &total);
        for (int g = g0; g < g1; ++g) {
            const uint64_t key = skey[g] & pmask;
            uint8_t keep = key > prefix;
            if (key == prefix) keep = rank++ < need;
            smask[g] = keep;
        }
    } else if (L.k == G) {
        for (int g = tid; g < G; g += kSelThreads) smask[g] = 1;
    }
    __syncthreads();

    // 3. mask and ascending kept list (ordered workgroup scan)
    uint32_t kept_local = 0;
    for (int g = g0; g < g1; ++g) kept_local += smask[g];
    uint32_t total;
    uint32_t pos = block_excl_scan(kept_local, scan_tmp, &total);
    for (int g = g0; g < g1; ++g) {
        L.mask[g] = smask[g];
        if (smask[g] && pos < (uint32_t)L.k) L.kept_idx[pos] = g;
        pos += smask[g];
    }

    // 4. per-column keep bytes for the apply pass
    if (L.colkeep) {
        const int64_t total_cols = (int64_t)L.groups * L.K;
        for (int64_t i = tid; i < total_cols; i += kSelThreads) {
            const int gc = (int)(i / L.K);
            const int j = (int)(i - (int64_t)gc * L.K);
            uint8_t sel = 1;
            if (L.kind == SA_SHAPE) sel = smask[j];
            else if (L.kind == SA_CHANNEL) sel = smask[j / L.CD];
            uint8_t al = L.allowed ? L.allowed[i] : 1;
            L.colkeep[i] = (sel && al) ? 1 : 0;
        }
    }
}

// ---------------------------------------------------------------- apply
// Z = v on kept entries, +0 elsewhere; fused: U' = v - Z, G = rho * ((W - Z) + U').
// Flat float4 stream over the layer; entry e sits at row e / K, column e % K.
struct ApplyLayer {
    const float *W;
    float *U;
    float *Z;
    float *G;
    const uint8_t *rowkeep;  // [A] or null
    const uint8_t *colkeep;  // [groups*K] or null
    const uint8_t *inmask;   // [groups*B] or null: column j of conv group gc is kept when
                             // inmask[gc * B + j / CD] is set
    FastDiv divK, divAg, divCD;
    int32_t n, K, B;
    float rho;
};
struct ApplyTab {
    ApplyLayer L[kTab];
    int32_t begin[kTab + 1];
    int32_t nl;
};

static_assert(sizeof(RowTab) < 8192 && sizeof(ColTab) < 8192 && sizeof(SelTab) < 8192 &&
                  sizeof(DualTab) < 8192 && sizeof(ApplyTab) < 8192 && sizeof(SgdTab) < 8192,
              "layer tables must fit the kernel-argument segment");

constexpr int kApplyThreads = 256;
constexpr int kApplyVec = 4;  // float4 per thread
constexpr int kApplyChunk = kApplyThreads * kApplyVec * 4;

__device__ inline void apply_one(const ApplyLayer &L, float w, float u, uint32_t row, uint32_t col, bool fused,
                                 float &z, float &un, float &g) {
    bool keep = true;
    if (L.rowkeep) keep = L.rowkeep[row] != 0;
    if (keep && L.colkeep) keep = L.colkeep[(int64_t)fdiv(row, L.divAg) * L.K + col] != 0;
    if (keep && L.inmask) keep = L.inmask[(int64_t)fdiv(row, L.divAg) * L.B + fdiv(col, L.divCD)] != 0;
    const float v = w + u;
    z = keep ? v : 0.0f;
    if (fused) {
        un = v - z;
        const float wz = w - z;
        const float s = wz + un;
        g = L.rho * s;
    }
}

__global__ __launch_bounds__(kApplyThreads) void k_apply(ApplyTab tab) {
    const int li = find_layer(tab.begin, tab.nl, blockIdx.x);
    const ApplyLayer &L = tab.L[li];
    const bool fused = L.G != nullptr;
    const int64_t c0 = (int64_t)(blockIdx.x - tab.begin[li]) * kApplyChunk;
    float4 xw[kApplyVec], xu[kApplyVec];
#pragma unroll
    for (int q = 0; q < kApplyVec; ++q) {
        const int64_t e = c0 + ((int64_t)q * kApplyThreads + threadIdx.x) * 4;
        if (e + 4 <= L.n) {
            xw[q] = *reinterpret_cast<const float4 *>(L.W + e);
            xu[q] = *reinterpret_cast<const float4 *>(L.U + e);
        }
    }
#pragma unroll
    for (int q = 0; q < kApplyVec; ++q) {
        const int64_t e = c0 + ((int64_t)q * kApplyThreads + threadIdx.x) * 4;
        if (e >= L.n) continue;
        if (e + 4 <= L.n) {
            uint32_t row = fdiv((uint32_t)e, L.divK);
            uint32_t col = (uint32_t)e - row * (uint32_t)L.K;
            float w[4] = {xw[q].x, xw[q].y, xw[q].z, xw[q].w};
            float u[4] = {xu[q].x, xu[q].y, xu[q].z, xu[q].w};
            float z[4], un[4], g[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                apply_one(L, w[i], u[i], row, col, fused, z[i], un[i], g[i]);
                if (++col == (uint32_t)L.K) {
                    col = 0;
                    ++row;
                }
            }
            // non-temporal stores: the outputs stream past the caches, which
            // keep W and U (read by the score pass just before) for the loads
            // above (measured 5% faster on the ResNet-50 step, 9% on 1 GB)
            nt_store4(L.Z + e, z);
            if (fused) {
                nt_store4(L.U + e, un);
                nt_store4(L.G + e, g);
            }
        } else {
            for (int64_t f = e; f < L.n; ++f) {
                uint32_t row = fdiv((uint32_t)f, L.divK);
                uint32_t col = (uint32_t)f - row * (uint32_t)L.K;
                float z, un = 0.f, g = 0.f;
                apply_one(L, L.W[f], L.U[f], row, col, fused, z, un, g);
                L.Z[f] = z;
                if (fused) {
                    L.U[f] = un;
                    L.G[f] = g;
                }
            }
        }
    }
}

// ---------------------------------------------------------------- element-wise
struct ElemState {
    uint32_t prefix;  // digits of T found so far; after the last pass, T itself
    uint32_t kk;      // rank of T among keys matching the prefix
    uint32_t gt;      // keys known to exceed T
    uint32_t pad;
};

struct ElemArgs {
    const float *W;
    float *U;
    float *Z;
    float *G;
    uint8_t *mask;
    int32_t *kept_idx;
    double *scores;          // [n] keys as |v| in binary64, or null
    const uint8_t *allowed;  // [groups*K] or null
    uint32_t *hist;          // [3][2048]
    ElemState *state;
    uint32_t *chunk_counts;  // [nchunks][2]: (gt, eq)
    uint32_t *chunk_prefix;  // [nchunks][2]: exclusive prefixes
    FastDiv divK;            // e -> row
    int32_t n, K, Ag, k, nchunks, vec;
    float rho;
};

// Is entry e inside the input-channel support?
__device__ inline bool elem_allowed(uint32_t e, const ElemArgs &a) {
    if (!a.allowed) return true;
    uint32_t row = fdiv(e, a.divK);
    uint32_t j = e - row * (uint32_t)a.K;
    return a.allowed[(int64_t)(row / a.Ag) * a.K + j] != 0;
}

// Key of entry e: |v| as binary32 bits (sign cleared); 0 outside the support.
__device__ inline uint32_t elem_key(float v, uint32_t e, const ElemArgs &a) {
    uint32_t key = __float_as_uint(v) & 0x7fffffffu;
    return elem_allowed(e, a) ? key : 0u;
}

__device__ inline void elem_load8(const ElemArgs &a, int64_t e0, float *w, float *v) {
    if (a.vec && e0 + 8 <= a.n) {
        float4 w0 = *reinterpret_cast<const float4 *>(a.W + e0);
        float4 w1 = *reinterpret_cast<const float4 *>(a.W + e0 + 4);
        float4 u0 = *reinterpret_cast<const float4 *>(a.U + e0);
        float4 u1 = *reinterpret_cast<const float4 *>(a.U + e0 + 4);
        w[0] = w0.x; w[1] = w0.y; w[2] = w0.z; w[3] = w0.w;
        w[4] = w1.x; w[5] = w1.y; w[6] = w1.z; w[7] = w1.w;
        v[0] = w0.x + u0.x; v[1] = w0.y + u0.y; v[2] = w0.z + u0.z; v[3] = w0.w + u0.w;
        v[4] = w1.x + u1.x; v[5] = w1.y + u1.y; v[6] = w1.z + u1.z; v[7] = w1.w + u1.w;
    } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            int64_t e = e0 + q;
            if (e < a.n) {
                w[q] = a.W[e];
                v[q] = w[q] + a.U[e];
            } else {
                w[q] = 0.f;
                v[q] = 0.f;
            }
        }
    }
}

__global__ void k_elem_init(ElemArgs a) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < 3 * 2048) a.hist[i] = 0;
    if (i == 0) {
        a.state->prefix = a.k > 0 ? 0u : 0x80000000u;  // k = 0: T above every key
        a.state->kk = (uint32_t)a.k;
        a.state->gt = 0;
        a.state->pad = 0;
    }
}

// Histogram of one digit of the keys that match the digits found so far.
// Digits: pass 0 = bits 30..20, pass 1 = bits 19..9, pass 2 = bits 8..0.
__global__ __launch_bounds__(kElemThreads) void k_elem_hist(ElemArgs a, int pass) {
    __shared__ uint32_t h[2048];
    for (int i = threadIdx.x; i < 2048; i += kElemThreads) h[i] = 0;
    __syncthreads();
    const uint32_t prefix = a.state->prefix;
    const int dshift = pass == 0 ? 20 : (pass == 1 ? 9 : 0);
    const uint32_t dmask = pass == 2 ? 0x1ffu : 0x7ffu;
    const int mshift = pass == 0 ? 31 : (pass == 1 ? 20 : 9);
    for (int c = blockIdx.x; c < a.nchunks; c += gridDim.x) {
        const int64_t e0 = (int64_t)c * kElemChunk + (int64_t)threadIdx.x * kElemPerThread;
        float w[8], v[8];
        elem_load8(a, e0, w, v);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (e0 + q >= a.n) break;
            uint32_t key = elem_key(v[q], (uint32_t)(e0 + q), a);
            if (pass == 0 || (key >> mshift) == prefix) atomicAdd(&h[(key >> dshift) & dmask], 1u);
        }
    }
    __syncthreads();
    uint32_t *gh = a.hist + pass * 2048;
    for (int i = threadIdx.x; i < 2048; i += kElemThreads)
        if (h[i]) atomicAdd(&gh[i], h[i]);
}

// Picks the digit holding the kk-th largest key (one wavefront).
__global__ void k_elem_find(ElemArgs a, int pass) {
    const int lane = threadIdx.x;
    const int bins = pass == 2 ? 512 : 2048;
    const int bits = pass == 2 ? 9 : 11;
    const int per = bins / kWave;
    const uint32_t *gh = a.hist + pass * 2048;
    const uint32_t kk = a.state->kk;
    const uint32_t prefix = a.state->prefix;
    uint32_t sum = 0;
    for (int q = 0; q < per; ++q) sum += gh[bins - 1 - lane * per - q];
    uint32_t incl = wave_incl_scan(sum);
    uint32_t excl = incl - sum;
    if (excl < kk && kk <= incl) {
        uint32_t above = excl;
        int d = 0;
        for (int q = 0; q < per; ++q) {
            int dig = bins - 1 - lane * per - q;
            uint32_t c = gh[dig];
            if (above + c >= kk) {
                d = dig;
                break;
            }
            above += c;
        }
        a.state->prefix = (prefix << bits) | (uint32_t)d;
        a.state->kk = kk - above;
        a.state->gt += above;
    }
}

// Per-chunk counts of keys above T and equal to T.
__global__ __launch_bounds__(kElemThreads) void k_elem_count(ElemArgs a) {
    __shared__ uint32_t red[2][kElemThreads / kWave];
    const int c = blockIdx.x;
    const uint32_t T = a.state->prefix;
    const int64_t e0 = (int64_t)c * kElemChunk + (int64_t)threadIdx.x * kElemPerThread;
    float w[8], v[8];
    elem_load8(a, e0, w, v);
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        if (e0 + q >= a.n) break;
        uint32_t key = elem_key(v[q], (uint32_t)(e0 + q), a);
        gt += key > T;
        eq += key == T;
    }
    gt = wave_sum_u32(gt);
    eq = wave_sum_u32(eq);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[0][wave] = gt;
        red[1][wave] = eq;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t g = 0, e = 0;
        for (int i = 0; i < kElemThreads / kWave; ++i) {
            g += red[0][i];
            e += red[1][i];
        }
        a.chunk_counts[2 * c] = g;
        a.chunk_counts[2 * c + 1] = e;
    }
}

// Exclusive prefixes of the per-chunk counts (one workgroup, chunk order).
__global__ __launch_bounds__(1024) void k_elem_scan(ElemArgs a) {
    __shared__ uint32_t tmp[1024 / kWave + 1];
    uint32_t carry_gt = 0, carry_eq = 0;
    for (int base = 0; base < a.nchunks; base += 1024) {
        const int c = base + threadIdx.x;
        uint32_t g = c < a.nchunks ? a.chunk_counts[2 * c] : 0u;
        uint32_t e = c < a.nchunks ? a.chunk_counts[2 * c + 1] : 0u;
        uint32_t tg, te;
        uint32_t pg = block_excl_scan(g, tmp, &tg);
        uint32_t pe = block_excl_scan(e, tmp, &te);
        if (c < a.nchunks) {
            a.chunk_prefix[2 * c] = carry_gt + pg;
            a.chunk_prefix[2 * c + 1] = carry_eq + pe;
        }
        carry_gt += tg;
        carry_eq += te;
    }
}

// Mask, ascending kept_idx, Z (+ fused U', G) for the non-structured set.
__global__ __launch_bounds__(kElemThreads) void k_elem_apply(ElemArgs a) {
    __shared__ uint32_t tmp[kElemThreads / kWave + 1];
    const int c = blockIdx.x;
    const uint32_t T = a.state->prefix;
    const uint32_t need = a.state->kk;  // ties at T kept overall (0 when k = 0)
    const uint32_t gt_before = a.chunk_prefix[2 * c];
    const uint32_t eq_before = a.chunk_prefix[2 * c + 1];
    const int64_t e0 = (int64_t)c * kElemChunk + (int64_t)threadIdx.x * kElemPerThread;
    float w[8], v[8];
    elem_load8(a, e0, w, v);
    uint32_t key[8];
    uint32_t eq = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        key[q] = (e0 + q < a.n) ? elem_key(v[q], (uint32_t)(e0 + q), a) : 0u;
        eq += (e0 + q < a.n) && key[q] == T;
    }
    uint32_t total;
    uint32_t eq_rank = eq_before + block_excl_scan(eq, tmp, &total);
    bool keep[8];
    uint32_t kept = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        keep[q] = false;
        if (e0 + q < a.n && a.k > 0) {
            if (key[q] > T) keep[q] = true;
            else if (key[q] == T) keep[q] = (eq_rank++ < need);
        }
        kept += keep[q];
    }
    const uint32_t kept_chunk_before = gt_before + min(eq_before, need);
    uint32_t pos = kept_chunk_before + block_excl_scan(kept, tmp, &total);
    const bool fused = a.G != nullptr;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int64_t e = e0 + q;
        if (e >= a.n) break;
        // a kept entry outside the support (score 0) still projects to 0
        const float z = (keep[q] && elem_allowed((uint32_t)e, a)) ? v[q] : 0.0f;
        a.Z[e] = z;
        a.mask[e] = keep[q] ? 1 : 0;
        if (a.scores) a.scores[e] = (double)__uint_as_float(key[q]);
        if (keep[q] && pos < (uint32_t)a.k) a.kept_idx[pos] = (int32_t)e;
        pos += keep[q] ? 1u : 0u;
        if (fused) {
            float un = v[q] - z;
            float wz = w[q] - z;
            float s = wz + un;
            a.U[e] = un;
            a.G[e] = a.rho * s;
        }
    }
}

// ---------------------------------------------------------------- dual
constexpr int kDualThreads = 256;
constexpr int kDualVecPerThread = 4;  // float4 per thread per workgroup pass
constexpr int kDualChunk = kDualThreads * kDualVecPerThread * 4;

// U <- (U + W) - Z;  G = rho * ((W - Z) + U)   (U new, or unchanged if !update)
__global__ __launch_bounds__(kDualThreads) void k_dual(DualTab tab) {
    const int li = find_layer(tab.begin, tab.nl, blockIdx.x);
    const DualLayer &L = tab.L[li];
    const int64_t c0 = (int64_t)(blockIdx.x - tab.begin[li]) * kDualChunk;
    const int n4 = L.n >> 2;
    // every load of the thread issued before any store; U and G are written
    // with the non-temporal hint (streamed past the caches: measured 72.7 ->
    // 56.9 us for the 23.45 M-weight ResNet-50 gradient pass)
    float4 w[kDualVecPerThread], z[kDualVecPerThread], uu[kDualVecPerThread];
#pragma unroll
    for (int u = 0; u < kDualVecPerThread; ++u) {
        const int64_t i = (c0 >> 2) + (int64_t)u * kDualThreads + threadIdx.x;
        if (i < n4) {
            w[u] = reinterpret_cast<const float4 *>(L.W)[i];
            z[u] = reinterpret_cast<const float4 *>(L.Z)[i];
            uu[u] = reinterpret_cast<const float4 *>(L.U)[i];
        }
    }
#pragma unroll
    for (int u = 0; u < kDualVecPerThread; ++u) {
        const int64_t i = (c0 >> 2) + (int64_t)u * kDualThreads + threadIdx.x;
        if (i < n4) {
            float wv[4] = {w[u].x, w[u].y, w[u].z, w[u].w}, zv[4] = {z[u].x, z[u].y, z[u].z, z[u].w};
            float uv[4] = {uu[u].x, uu[u].y, uu[u].z, uu[u].w}, gv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (L.update) {
                    float s = uv[e] + wv[e];
                    uv[e] = s - zv[e];
                }
                float wz = wv[e] - zv[e];
                float t = wz + uv[e];
                gv[e] = L.rho * t;
            }
            if (L.update) nt_store4(reinterpret_cast<float *>(L.U) + 4 * i, uv);
            if (L.G) nt_store4(reinterpret_cast<float *>(L.G) + 4 * i, gv);
        }
    }
    // scalar tail (n % 4 entries), handled by the layer's first workgroup
    if (blockIdx.x == tab.begin[li] && threadIdx.x < (L.n & 3)) {
        const int64_t e = (int64_t)n4 * 4 + threadIdx.x;
        float u = L.U[e];
        if (L.update) {
            float s = u + L.W[e];
            u = s - L.Z[e];
            L.U[e] = u;
        }
        if (L.G) {
            float wz = L.W[e] - L.Z[e];
            float t = wz + u;
            L.G[e] = L.rho * t;
        }
    }
}

// ---------------------------------------------------------------- SGD step
constexpr int kSgdThreads = 256;
constexpr int kSgdVecPerThread = 4;
constexpr int kSgdChunk = kSgdThreads * kSgdVecPerThread * 4;

__device__ inline bool sgd_keep(const SgdLayer &L, uint32_t e) {
    if (!L.mask) return true;
    uint32_t g = e;
    if (L.kind != SA_ELEMENT) {
        const uint32_t a = fdiv(e, L.divK);
        const uint32_t j = e - a * L.divK.d;  // column (b*C + c)*D + d
        g = L.kind == SA_FILTER ? a : L.kind == SA_CHANNEL ? fdiv(j, L.divCD) : j;
    }
    return L.mask[g] != 0;
}

// t = Gf + rho * ((W - Z) + U) (or Gf);  W <- keep ? W - lr * t : +0
__device__ inline float sgd_one(const SgdLayer &L, float w, float gf, float z, float u, bool keep) {
    float t = gf;
    if (L.Z) {
        const float d = w - z;
        const float sum = d + u;
        const float r = L.rho * sum;
        t = gf + r;
    }
    const float q = L.lr * t;
    return keep ? w - q : 0.0f;
}

__global__ __launch_bounds__(kSgdThreads) void k_sgd(SgdTab tab) {
    const int li = find_layer(tab.begin, tab.nl, blockIdx.x);
    const SgdLayer &L = tab.L[li];
    const int64_t c0 = (int64_t)(blockIdx.x - tab.begin[li]) * kSgdChunk;
    const int n4 = L.n >> 2;
#pragma unroll
    for (int v = 0; v < kSgdVecPerThread; ++v) {
        const int64_t i = (c0 >> 2) + (int64_t)v * kSgdThreads + threadIdx.x;
        if (i < n4) {
            const float4 w = reinterpret_cast<const float4 *>(L.W)[i];
            const float4 g = reinterpret_cast<const float4 *>(L.Gf)[i];
            float4 z = make_float4(0.f, 0.f, 0.f, 0.f), u = z;
            if (L.Z) {
                z = reinterpret_cast<const float4 *>(L.Z)[i];
                u = reinterpret_cast<const float4 *>(L.U)[i];
            }
            const uint32_t e = (uint32_t)i * 4u;
            float4 o;
            o.x = sgd_one(L, w.x, g.x, z.x, u.x, sgd_keep(L, e));
            o.y = sgd_one(L, w.y, g.y, z.y, u.y, sgd_keep(L, e + 1));
            o.z = sgd_one(L, w.z, g.z, z.z, u.z, sgd_keep(L, e + 2));
            o.w = sgd_one(L, w.w, g.w, z.w, u.w, sgd_keep(L, e + 3));
            reinterpret_cast<float4 *>(L.W)[i] = o;
        }
    }
    // scalar tail (n % 4 entries), handled by the layer's first workgroup
    if (blockIdx.x == tab.begin[li] && threadIdx.x < (L.n & 3)) {
        const uint32_t e = (uint32_t)n4 * 4u + threadIdx.x;
        const float z = L.Z ? L.Z[e] : 0.f, u = L.Z ? L.U[e] : 0.f;
        L.W[e] = sgd_one(L, L.W[e], L.Gf[e], z, u, sgd_keep(L, e));
    }
}

// ---------------------------------------------------------------- host planning
struct LayerPlan {
    int64_t G;
    int K, CD, Ag, R, rchunks, ritems, nbands, ctiles, vec, nchunks;
    size_t off_scores, off_rowpart, off_partials, off_allowed, off_colkeep, off_elem;
    size_t end;
};

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

void plan_layer(const sa_project_desc &d, size_t start, LayerPlan &p) {
    p.G = n_groups(d);
    p.K = (int)(d.B * d.C * d.D);
    p.CD = (int)(d.C * d.D);
    p.Ag = (int)(d.A / d.groups);
    p.vec = (p.K % 4 == 0) ? 1 : 0;
    // filter scores: work items of one wavefront each
    const int K4 = p.K / 4;
    p.R = !p.vec ? 1 : (K4 <= kWave ? 4 : (K4 <= 2 * kWave ? 2 : 1));
    p.rchunks = (p.vec && p.R == 1) ? (K4 + 4 * kWave - 1) / (4 * kWave) : 1;
    p.ritems = !p.vec ? (int)d.A : (p.R > 1 ? (int)((d.A + p.R - 1) / p.R) : (int)d.A * p.rchunks);
    p.nbands = (int)((d.A + kColBand - 1) / kColBand);
    const int cols_per_block = (kColThreads / kColSlices) * (p.vec ? 4 : 1);
    p.ctiles = (p.K + cols_per_block - 1) / cols_per_block;
    const int64_t n = d.A * d.B * d.C * d.D;
    p.nchunks = (int)((n + kElemChunk - 1) / kElemChunk);
    size_t off = align256(start);
    p.off_scores = p.off_rowpart = p.off_partials = p.off_allowed = p.off_colkeep = p.off_elem = SIZE_MAX;
    if (d.kind != SA_ELEMENT && !d.scores) {
        p.off_scores = off;
        off = align256(off + sizeof(double) * p.G);
    }
    if (d.kind == SA_FILTER && p.rchunks > 1) {
        p.off_rowpart = off;
        off = align256(off + sizeof(double) * (size_t)d.A * p.rchunks);
    }
    if (d.kind == SA_CHANNEL || d.kind == SA_SHAPE) {
        p.off_partials = off;
        off = align256(off + sizeof(double) * (size_t)p.nbands * p.K);
    }
    if (d.in_ch_mask && d.kind != SA_FILTER) {
        p.off_allowed = off;
        off = align256(off + (size_t)d.groups * p.K);
    }
    if (d.kind == SA_CHANNEL || d.kind == SA_SHAPE) {
        p.off_colkeep = off;
        off = align256(off + (size_t)d.groups * p.K);
    }
    if (d.kind == SA_ELEMENT) {
        p.off_elem = off;
        off = align256(off + sizeof(uint32_t) * 3 * 2048 + sizeof(ElemState) +
                       sizeof(uint32_t) * 4 * (size_t)p.nchunks + 256);
    }
    p.end = off;
}

template <typename T>
T *ws_at(void *ws, size_t off) {
    return reinterpret_cast<T *>(static_cast<char *>(ws) + off);
}

int launch_check(const char *what) { return check_hip(hipGetLastError(), what); }

}  // namespace
}  // namespace sa

using namespace sa;

extern "C" size_t structadmm_project_workspace(const sa_project_desc *layers, int n_layers) {
    if (!layers || n_layers <= 0) return 0;
    size_t off = 0;
    for (int i = 0; i < n_layers; ++i) {
        if (validate_project(layers[i], i) != SA_OK) {
            clear_error();
            return 0;
        }
        LayerPlan p;
        plan_layer(layers[i], off, p);
        off = p.end;
    }
    return off;
}

namespace sa {
namespace {

// Scratch of structadmm_project_noalloc: one copy per GPU, in the code
// object's device memory, held until the process ends.  Host code never uses
// the symbol itself as an address: the device address of each GPU's copy
// comes from hipGetSymbolAddress with that GPU current.
__device__ __align__(256) uint8_t scratch[SA_PROJECT_NOALLOC_BYTES];

constexpr int kMaxDevices = 64;

// Device address of the current GPU's scratch (nullptr and an error set on failure).
void *noalloc_scratch() {
    static std::mutex mu;
    static void *ptr[kMaxDevices] = {};
    int dev = 0;
    if (check_hip(hipGetDevice(&dev), "project_noalloc: current device")) return nullptr;
    if (dev < 0 || dev >= kMaxDevices) {
        fail(SA_E_UNSUPPORTED, "project_noalloc: device index %d beyond %d", dev, kMaxDevices);
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(mu);
    if (!ptr[dev]) {
        void *p = nullptr;
        if (check_hip(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "project_noalloc: scratch address")) return nullptr;
        ptr[dev] = p;
    }
    return ptr[dev];
}

int project_impl(const sa_project_desc *layers, int n_layers, void *ws, size_t ws_bytes, hipStream_t stream);

}  // namespace
}  // namespace sa

extern "C" int structadmm_project(const sa_project_desc *layers, int n_layers, void *ws,
                                  size_t ws_bytes, hipStream_t stream) {
    clear_error();
    return project_impl(layers, n_layers, ws, ws_bytes, stream);
}

extern "C" int structadmm_project_noalloc(const sa_project_desc *layers, int n_layers, hipStream_t stream) {
    clear_error();
    if (!layers || n_layers <= 0) return fail(SA_E_ARG, "project: layers must be a non-empty array");
    size_t need = 0;
    for (int i = 0; i < n_layers; ++i) {
        if (int rc = validate_project(layers[i], i)) return rc;
        LayerPlan p;
        plan_layer(layers[i], need, p);
        need = p.end;
    }
    if (need > (size_t)SA_PROJECT_NOALLOC_BYTES)
        return fail(SA_E_WORKSPACE, "project_noalloc: these layers need %zu bytes of scratch, more than the %zu "
                    "the library holds (use structadmm_project with a workspace)", need,
                    (size_t)SA_PROJECT_NOALLOC_BYTES);
    void *ws = need > 0 ? noalloc_scratch() : nullptr;
    if (need > 0 && !ws) return SA_E_HIP;
    return project_impl(layers, n_layers, ws, SA_PROJECT_NOALLOC_BYTES, stream);
}

namespace sa {
namespace {

int project_impl(const sa_project_desc *layers, int n_layers, void *ws, size_t ws_bytes, hipStream_t stream) {
    if (!layers || n_layers <= 0) return fail(SA_E_ARG, "project: layers must be a non-empty array");
    std::vector<LayerPlan> plan(n_layers);
    size_t off = 0;
    for (int i = 0; i < n_layers; ++i) {
        int rc = validate_project(layers[i], i);
        if (rc) return rc;
        plan_layer(layers[i], off, plan[i]);
        off = plan[i].end;
    }
    if (off > 0) {
        if (!ws) return fail(SA_E_WORKSPACE, "project: workspace of %zu bytes required", off);
        if (ws_bytes < off)
            return fail(SA_E_WORKSPACE, "project: workspace %zu bytes < required %zu", ws_bytes, off);
        if (!aligned(ws, 256)) return fail(SA_E_ALIGN, "project: workspace must be 256-byte aligned");
    }
    // dependency levels: a layer whose in_ch_mask is an earlier layer's mask runs after it
    std::vector<int> level(n_layers, 0);
    int max_level = 0;
    for (int i = 0; i < n_layers; ++i) {
        for (int j = 0; j < i; ++j)
            if (layers[i].in_ch_mask && (const void *)layers[i].in_ch_mask == (const void *)layers[j].mask)
                level[i] = std::max(level[i], level[j] + 1);
        max_level = std::max(max_level, level[i]);
    }

    auto fill_row = [&](int i, RowLayer &R) {
        const sa_project_desc &d = layers[i];
        const LayerPlan &p = plan[i];
        R.W = d.W;
        R.U = d.U;
        // filter sets read their support straight from the input-channel mask;
        // the other sets use its per-column expansion
        R.allowed = d.in_ch_mask && d.kind != SA_FILTER ? ws_at<uint8_t>(ws, p.off_allowed) : nullptr;
        R.inmask = d.kind == SA_FILTER ? d.in_ch_mask : nullptr;
        R.B = (int)d.B;
        R.divCD = make_fastdiv((uint32_t)p.CD);
        R.scores = d.scores ? d.scores : (p.off_scores != SIZE_MAX ? ws_at<double>(ws, p.off_scores) : nullptr);
        R.A = (int)d.A;
        R.K = p.K;
        R.Ag = p.Ag;
        R.R = p.R;
        R.nchunk = p.rchunks;
        R.rowpart = p.off_rowpart != SIZE_MAX ? ws_at<double>(ws, p.off_rowpart) : nullptr;
        R.vec = p.vec;
        R.rho = d.rho;
    };

    for (int lv = 0; lv <= max_level; ++lv) {
        std::vector<int> ids;
        for (int i = 0; i < n_layers; ++i)
            if (level[i] == lv) ids.push_back(i);

        // allowed bytes for layers with a channel support (filter sets read
        // the mask itself)
        for (int i : ids) {
            const sa_project_desc &d = layers[i];
            if (!d.in_ch_mask || d.kind == SA_FILTER) continue;
            const LayerPlan &p = plan[i];
            int64_t total = (int64_t)d.groups * p.K;
            int blocks = (int)std::min<int64_t>(1024, (total + 255) / 256);
            hipLaunchKernelGGL(k_expand_allowed, dim3(blocks), dim3(256), 0, stream, d.in_ch_mask,
                               ws_at<uint8_t>(ws, p.off_allowed), d.groups, (int)d.B, p.CD, p.K);
            if (int rc = launch_check("k_expand_allowed")) return rc;
        }


        // filter scores
        {
            std::vector<int> f;
            for (int i : ids)
                if (layers[i].kind == SA_FILTER) f.push_back(i);
            for (size_t s = 0; s < f.size(); s += kTab) {
                RowTab tab;
                memset(&tab, 0, sizeof tab);
                int blocks = 0;
                tab.nl = (int)std::min<size_t>(kTab, f.size() - s);
                for (int t = 0; t < tab.nl; ++t) {
                    fill_row(f[s + t], tab.L[t]);
                    tab.begin[t] = blocks;
                    blocks += (plan[f[s + t]].ritems + kRowItems * (kRowThreads / kWave) - 1) /
                              (kRowItems * (kRowThreads / kWave));
                }
                tab.begin[tab.nl] = blocks;
                hipLaunchKernelGGL(k_row_scores, dim3(blocks), dim3(kRowThreads), 0, stream, tab);
                if (int rc = launch_check("k_row_scores")) return rc;
            }
        }
        // channel / shape column partials
        {
            std::vector<int> c;
            for (int i : ids)
                if (layers[i].kind == SA_CHANNEL || layers[i].kind == SA_SHAPE) c.push_back(i);
            for (size_t s = 0; s < c.size(); s += kTab) {
                ColTab tab;
                memset(&tab, 0, sizeof tab);
                int blocks = 0;
                tab.nl = (int)std::min<size_t>(kTab, c.size() - s);
                for (int t = 0; t < tab.nl; ++t) {
                    const sa_project_desc &d = layers[c[s + t]];
                    const LayerPlan &p = plan[c[s + t]];
                    ColLayer &L = tab.L[t];
                    L.W = d.W;
                    L.U = d.U;
                    L.allowed = d.in_ch_mask ? ws_at<uint8_t>(ws, p.off_allowed) : nullptr;
                    L.partials = ws_at<double>(ws, p.off_partials);
                    L.A = (int)d.A;
                    L.K = p.K;
                    L.Ag = p.Ag;
                    L.nbands = p.nbands;
                    L.ctiles = p.ctiles;
                    L.vec = p.vec;
                    tab.begin[t] = blocks;
                    blocks += p.nbands * p.ctiles;
                }
                tab.begin[tab.nl] = blocks;
                hipLaunchKernelGGL(k_col_partials, dim3(blocks), dim3(kColThreads), 0, stream, tab);
                if (int rc = launch_check("k_col_partials")) return rc;
            }
        }
        // selection for every structured layer
        {
            std::vector<int> sl;
            for (int i : ids)
                if (layers[i].kind != SA_ELEMENT) sl.push_back(i);
            for (size_t s = 0; s < sl.size(); s += kTab) {
                SelTab tab;
                memset(&tab, 0, sizeof tab);
                tab.nl = (int)std::min<size_t>(kTab, sl.size() - s);
                for (int t = 0; t < tab.nl; ++t) {
                    const sa_project_desc &d = layers[sl[s + t]];
                    const LayerPlan &p = plan[sl[s + t]];
                    SelLayer &L = tab.L[t];
                    L.partials = p.off_partials != SIZE_MAX ? ws_at<double>(ws, p.off_partials) : nullptr;
                    L.scores = d.scores ? d.scores : ws_at<double>(ws, p.off_scores);
                    L.rowpart = p.off_rowpart != SIZE_MAX ? ws_at<double>(ws, p.off_rowpart) : nullptr;
                    L.nchunk = p.rchunks;
                    L.mask = d.mask;
                    L.kept_idx = d.kept_idx;
                    L.colkeep = p.off_colkeep != SIZE_MAX ? ws_at<uint8_t>(ws, p.off_colkeep) : nullptr;
                    L.allowed = p.off_allowed != SIZE_MAX ? ws_at<uint8_t>(ws, p.off_allowed) : nullptr;
                    L.kind = d.kind;
                    L.G = (int)p.G;
                    L.k = (int)d.k;
                    L.K = p.K;
                    L.CD = p.CD;
                    L.nbands = p.nbands;
                    L.groups = d.groups;
                }
                hipLaunchKernelGGL(k_select, dim3(tab.nl), dim3(kSelThreads), 0, stream, tab);
                if (int rc = launch_check("k_select")) return rc;
            }
        }
        // element-wise layers
        for (int i : ids) {
            const sa_project_desc &d = layers[i];
            if (d.kind != SA_ELEMENT) continue;
            const LayerPlan &p = plan[i];
            ElemArgs a;
            memset(&a, 0, sizeof a);
            a.W = d.W;
            a.U = d.U;
            a.Z = d.Z;
            a.G = d.G;
            a.mask = d.mask;
            a.kept_idx = d.kept_idx;
            a.scores = d.scores;
            a.allowed = d.in_ch_mask ? ws_at<uint8_t>(ws, p.off_allowed) : nullptr;
            char *eb = ws_at<char>(ws, p.off_elem);
            a.hist = reinterpret_cast<uint32_t *>(eb);
            a.state = reinterpret_cast<ElemState *>(eb + sizeof(uint32_t) * 3 * 2048);
            a.chunk_counts = reinterpret_cast<uint32_t *>(eb + sizeof(uint32_t) * 3 * 2048 + 256);
            a.chunk_prefix = a.chunk_counts + 2 * (size_t)p.nchunks;
            a.divK = make_fastdiv((uint32_t)p.K);
            a.n = (int32_t)(d.A * d.B * d.C * d.D);
            a.K = p.K;
            a.Ag = p.Ag;
            a.k = (int32_t)d.k;
            a.nchunks = p.nchunks;
            a.vec = 1;  // n is a multiple of 4 only sometimes; elem_load8 checks the tail
            a.rho = d.rho;
            hipLaunchKernelGGL(k_elem_init, dim3((3 * 2048 + 255) / 256), dim3(256), 0, stream, a);
            if (int rc = launch_check("k_elem_init")) return rc;
            if (d.k > 0) {
                const int hb = std::min(p.nchunks, kElemHistBlocks);
                for (int pass = 0; pass < 3; ++pass) {
                    hipLaunchKernelGGL(k_elem_hist, dim3(hb), dim3(kElemThreads), 0, stream, a, pass);
                    if (int rc = launch_check("k_elem_hist")) return rc;
                    hipLaunchKernelGGL(k_elem_find, dim3(1), dim3(kWave), 0, stream, a, pass);
                    if (int rc = launch_check("k_elem_find")) return rc;
                }
            }
            hipLaunchKernelGGL(k_elem_count, dim3(p.nchunks), dim3(kElemThreads), 0, stream, a);
            if (int rc = launch_check("k_elem_count")) return rc;
            hipLaunchKernelGGL(k_elem_scan, dim3(1), dim3(1024), 0, stream, a);
            if (int rc = launch_check("k_elem_scan")) return rc;
            hipLaunchKernelGGL(k_elem_apply, dim3(p.nchunks), dim3(kElemThreads), 0, stream, a);
            if (int rc = launch_check("k_elem_apply")) return rc;
        }
    }
    // apply for every structured layer, all levels at once: a level only needs
    // the masks of the levels before it, never their Z / U / G
    {
        std::vector<int> sl;
        for (int i = 0; i < n_layers; ++i)
            if (layers[i].kind != SA_ELEMENT) sl.push_back(i);
        for (size_t s = 0; s < sl.size(); s += kTab) {
            ApplyTab tab;
            memset(&tab, 0, sizeof tab);
            int blocks = 0;
            tab.nl = (int)std::min<size_t>(kTab, sl.size() - s);
            for (int t = 0; t < tab.nl; ++t) {
                RowLayer R;
                fill_row(sl[s + t], R);
                const sa_project_desc &d = layers[sl[s + t]];
                ApplyLayer &L = tab.L[t];
                L.W = R.W;
                L.U = R.U;
                L.Z = d.Z;
                L.G = d.G;
                L.rowkeep = d.kind == SA_FILTER ? d.mask : nullptr;
                L.colkeep = d.kind == SA_FILTER ? nullptr : ws_at<uint8_t>(ws, plan[sl[s + t]].off_colkeep);
                L.inmask = R.inmask;
                L.B = R.B;
                L.divCD = R.divCD;
                L.divK = make_fastdiv((uint32_t)R.K);
                L.divAg = make_fastdiv((uint32_t)R.Ag);
                L.n = (int32_t)(d.A * d.B * d.C * d.D);
                L.K = R.K;
                L.rho = R.rho;
                tab.begin[t] = blocks;
                blocks += (int)((L.n + kApplyChunk - 1) / kApplyChunk);
            }
            tab.begin[tab.nl] = blocks;
            hipLaunchKernelGGL(k_apply, dim3(blocks), dim3(kApplyThreads), 0, stream, tab);
            if (int rc = launch_check("k_apply")) return rc;
        }
    }
    return SA_OK;
}

}  // namespace
}  // namespace sa

extern "C" int structadmm_dual_update(const sa_dual_desc *layers, int n_layers, hipStream_t stream) {
    clear_error();
    if (!layers || n_layers <= 0) return fail(SA_E_ARG, "dual_update: layers must be a non-empty array");
    for (int i = 0; i < n_layers; ++i)
        if (int rc = validate_dual(layers[i], i)) return rc;
    for (int s = 0; s < n_layers; s += kTab) {
        DualTab tab;
        memset(&tab, 0, sizeof tab);
        tab.nl = std::min(kTab, n_layers - s);
        int blocks = 0;
        for (int t = 0; t < tab.nl; ++t) {
            const sa_dual_desc &d = layers[s + t];
            DualLayer &L = tab.L[t];
            L.W = d.W;
            L.Z = d.Z;
            L.U = d.U;
            L.G = d.G;
            L.n = (int32_t)d.n;
            L.update = d.update_dual ? 1 : 0;
            L.rho = d.rho;
            tab.begin[t] = blocks;
            blocks += (int)std::max<int64_t>(1, (d.n + kDualChunk - 1) / kDualChunk);
        }
        tab.begin[tab.nl] = blocks;
        hipLaunchKernelGGL(k_dual, dim3(blocks), dim3(kDualThreads), 0, stream, tab);
        if (int rc = launch_check("k_dual")) return rc;
    }
    return SA_OK;
}

extern "C" int structadmm_sgd_step(const sa_sgd_desc *layers, int n_layers, hipStream_t stream) {
    clear_error();
    if (!layers || n_layers <= 0) return fail(SA_E_ARG, "sgd_step: layers must be a non-empty array");
    for (int i = 0; i < n_layers; ++i)
        if (int rc = validate_sgd(layers[i], i)) return rc;
    for (int s = 0; s < n_layers; s += kTab) {
        SgdTab tab;
        memset(&tab, 0, sizeof tab);
        tab.nl = std::min(kTab, n_layers - s);
        int blocks = 0;
        for (int t = 0; t < tab.nl; ++t) {
            const sa_sgd_desc &d = layers[s + t];
            SgdLayer &L = tab.L[t];
            const int64_t n = d.A * d.B * d.C * d.D;
            L.W = d.W;
            L.Gf = d.Gf;
            L.Z = d.Z;
            L.U = d.U;
            L.mask = d.mask;
            L.n = (int32_t)n;
            L.kind = d.kind;
            L.divK = make_fastdiv((uint32_t)(d.B * d.C * d.D));
            L.divCD = make_fastdiv((uint32_t)(d.C * d.D));
            L.rho = d.rho;
            L.lr = d.lr;
            tab.begin[t] = blocks;
            blocks += (int)std::max<int64_t>(1, (n + kSgdChunk - 1) / kSgdChunk);
        }
        tab.begin[tab.nl] = blocks;
        hipLaunchKernelGGL(k_sgd, dim3(blocks), dim3(kSgdThreads), 0, stream, tab);
        if (int rc = launch_check("k_sgd")) return rc;
    }
    return SA_OK;
}
