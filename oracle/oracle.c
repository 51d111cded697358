/*
 * StructADMM oracle: a plain, slow CPU statement of what the hot path computes.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  The GPU library never
 * links, includes or calls it and the two share no source: no headers, no
 * helpers, no tables.
 *
 * Paper: "StructADMM: A Systematic, High-Efficiency Framework of Structured
 * Weight Pruning for DNNs" (arXiv 1807.11091).
 *   - Section 3 defines the weight tensor W in R^{A x B x C x D}, the slices
 *     X[a,:,:,:] (filter), X[:,b,:,:] (channel), X[:,b,c,d] (filter shape)
 *     and the four constraint sets (filter-, channel-, shape-wise and
 *     non-structured sparsity).
 *   - Section 4, eq. (3) and the line under it: the W-subproblem's quadratic
 *     term rho/2 ||W - Z + U||_F^2 and the dual update U^k = U^{k-1} + W^k - Z^k.
 *   - Section 4, eq. (4) and "Solving the second subproblem": Z is the
 *     Euclidean projection of W + U onto S, obtained by scoring every group
 *     with its squared Frobenius norm (or every element by its magnitude),
 *     keeping the largest ones and zeroing the rest.
 *   - Section 3, "Combination of structured sparsities": filter pruning
 *     removes GEMM rows, channel / shape pruning removes GEMM columns; the
 *     CONV then runs as a full GEMM with fewer rows / columns.
 *
 * Readings where the paper is silent (all documented in the design notes):
 *   - v = fl32(w + u) is one IEEE binary32 add; group scores accumulate
 *     (double)v * (double)v in binary64; element keys are |v|.
 *   - exactly k groups are kept; ties at the k-th key go to the lowest index.
 *   - an optional input-channel support (in_ch_mask) forces zeros on the
 *     masked (conv group, channel) slices; the projection onto the
 *     intersection scores only the unmasked entries.
 *   - the fused step returns U' = fl32(v - Z) and G = fl32(rho * fl32(fl32(W - Z) + U')).
 *   - the compacted matrix of a conv group has the group's kept filters as
 *     rows (ascending) and its kept (channel, tap) pairs as columns in the
 *     ascending order of the flattened GEMM column index j = (b*C + c)*D + d
 *     of Section 3's [A, B*C*D] view; its entries are Z rounded to bfloat16
 *     (round to nearest even).  The paper fixes no other column order: an
 *     implementation may permute the columns of a group (the GEMM is the same
 *     up to a permutation of its reduction index), and a comparison with this
 *     oracle matches columns by their (channel, tap) pair.
 *   - CONV is cross-correlation with zero padding, no bias, no dilation.
 *
 * Everything here is straight loops with no blocking, fusion or reordering.
 * Floating point is binary32 where the method's tensors are binary32 and
 * binary64 for every accumulation.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_FILTER = 0, OR_CHANNEL = 1, OR_SHAPE = 2, OR_ELEMENT = 3 };

/* Number of groups of each constraint set (Section 3). */
int64_t oracle_n_groups(int64_t A, int64_t B, int64_t C, int64_t D, int32_t kind)
{
    switch (kind) {
    case OR_FILTER: return A;
    case OR_CHANNEL: return B;
    case OR_SHAPE: return B * C * D;
    case OR_ELEMENT: return A * B * C * D;
    default: return -1;
    }
}

/* The group that weight (a, b, c, d) belongs to (Section 3 slice notation). */
static int64_t group_of(int64_t a, int64_t b, int64_t c, int64_t d,
                        int64_t B, int64_t C, int64_t D, int32_t kind)
{
    switch (kind) {
    case OR_FILTER: return a;
    case OR_CHANNEL: return b;
    case OR_SHAPE: return (b * C + c) * D + d;
    default: return ((a * B + b) * C + c) * D + d;
    }
}

/* Is weight (a, b, .., ..) inside the fixed input-channel support?  The
 * support is given per (conv group, channel) as in_ch_mask[gc * B + b]. */
static int channel_allowed(const uint8_t *in_ch_mask, int64_t a, int64_t b,
                           int64_t A, int64_t B, int32_t groups)
{
    if (!in_ch_mask)
        return 1;
    int64_t gc = a / (A / groups);
    return in_ch_mask[gc * B + b] != 0;
}

/* Step 1 of the Z-update (Section 4): V = W + U and the score of every group,
 * O_g = ||V_g||_F^2 for the structured sets, |v| for the non-structured set. */
void oracle_scores(int64_t A, int64_t B, int64_t C, int64_t D, int32_t groups, int32_t kind,
                   const float *W, const float *U, const uint8_t *in_ch_mask,
                   float *V, double *score)
{
    int64_t G = oracle_n_groups(A, B, C, D, kind);
    for (int64_t g = 0; g < G; ++g)
        score[g] = 0.0;
    for (int64_t a = 0; a < A; ++a)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t c = 0; c < C; ++c)
                for (int64_t d = 0; d < D; ++d) {
                    int64_t e = ((a * B + b) * C + c) * D + d;
                    float v = W[e] + U[e];
                    V[e] = v;
                    if (!channel_allowed(in_ch_mask, a, b, A, B, groups))
                        continue;
                    int64_t g = group_of(a, b, c, d, B, C, D, kind);
                    if (kind == OR_ELEMENT)
                        score[g] = fabs((double)v);
                    else
                        score[g] += (double)v * (double)v;
                }
}

typedef struct {
    double key;
    int64_t idx;
} keyed;

/* Larger key first; equal keys by ascending index. */
static int cmp_keyed(const void *pa, const void *pb)
{
    const keyed *x = (const keyed *)pa, *y = (const keyed *)pb;
    if (x->key > y->key) return -1;
    if (x->key < y->key) return 1;
    if (x->idx < y->idx) return -1;
    if (x->idx > y->idx) return 1;
    return 0;
}

/* Step 2: keep the k groups with the largest scores (Section 4); exactly k
 * are kept, ties at the boundary go to the lowest group index.
 * mask[g] = 1 for kept groups; kept_idx lists them in ascending order. */
int oracle_select(int64_t G, const double *key, int64_t k, uint8_t *mask, int32_t *kept_idx)
{
    if (k < 0 || k > G)
        return -1;
    keyed *order = (keyed *)malloc(sizeof(keyed) * (size_t)(G > 0 ? G : 1));
    if (!order)
        return -2;
    for (int64_t g = 0; g < G; ++g) {
        order[g].key = key[g];
        order[g].idx = g;
    }
    qsort(order, (size_t)G, sizeof(keyed), cmp_keyed);
    for (int64_t g = 0; g < G; ++g)
        mask[g] = 0;
    for (int64_t r = 0; r < k; ++r)
        mask[order[r].idx] = 1;
    int64_t j = 0;
    for (int64_t g = 0; g < G; ++g)
        if (mask[g])
            kept_idx[j++] = (int32_t)g;
    free(order);
    return 0;
}

/* The Z-update of Section 4 for one layer: Z = Proj_S(W + U).
 * With G != NULL it also takes the dual update of Section 4 with the same W
 * (U' = V - Z, written to U_out, which may alias U) and the gradient of the
 * quadratic term of eq. (3), G = rho * ((W - Z) + U').
 * scores may be NULL.  Returns 0, or a negative value on bad arguments. */
int oracle_project(int64_t A, int64_t B, int64_t C, int64_t D, int32_t groups, int32_t kind,
                   int64_t k, const float *W, const float *U, const uint8_t *in_ch_mask,
                   float rho, float *Z, uint8_t *mask, int32_t *kept_idx, double *scores,
                   float *U_out, float *Gout)
{
    if (A <= 0 || B <= 0 || C <= 0 || D <= 0 || groups <= 0 || A % groups != 0)
        return -1;
    int64_t n = A * B * C * D;
    int64_t G = oracle_n_groups(A, B, C, D, kind);
    if (G < 0 || k < 0 || k > G)
        return -1;
    float *V = (float *)malloc(sizeof(float) * (size_t)n);
    double *sc = scores ? scores : (double *)malloc(sizeof(double) * (size_t)G);
    if (!V || !sc)
        return -2;
    oracle_scores(A, B, C, D, groups, kind, W, U, in_ch_mask, V, sc);
    int rc = oracle_select(G, sc, k, mask, kept_idx);
    if (rc == 0) {
        for (int64_t a = 0; a < A; ++a)
            for (int64_t b = 0; b < B; ++b)
                for (int64_t c = 0; c < C; ++c)
                    for (int64_t d = 0; d < D; ++d) {
                        int64_t e = ((a * B + b) * C + c) * D + d;
                        int64_t g = group_of(a, b, c, d, B, C, D, kind);
                        int keep = mask[g] && channel_allowed(in_ch_mask, a, b, A, B, groups);
                        Z[e] = keep ? V[e] : 0.0f;
                    }
        if (Gout) {
            for (int64_t e = 0; e < n; ++e) {
                float u_new = V[e] - Z[e];
                float w_minus_z = W[e] - Z[e];
                float s = w_minus_z + u_new;
                Gout[e] = rho * s;
                U_out[e] = u_new;
            }
        }
    }
    if (!scores)
        free(sc);
    free(V);
    return rc;
}

/* Dual update U <- U + W - Z (Section 4, under eq. (3)) and the gradient of
 * rho/2 ||W - Z + U||_F^2 with respect to W, G = rho * ((W - Z) + U).
 * update_dual = 0 leaves U unchanged (the per-SGD-step gradient). G may be NULL. */
void oracle_dual_update(int64_t n, const float *W, const float *Z, float *U, float rho,
                        float *Gout, int32_t update_dual)
{
    for (int64_t e = 0; e < n; ++e) {
        float u = U[e];
        if (update_dual) {
            float u_plus_w = u + W[e];
            u = u_plus_w - Z[e];
            U[e] = u;
        }
        if (Gout) {
            float w_minus_z = W[e] - Z[e];
            float s = w_minus_z + u;
            Gout[e] = rho * s;
        }
    }
}

/* One SGD step of the W-subproblem (Section 4, eq. (3)) or of masked
 * retraining ("Masked mapping and retraining": pruned weights stay zero):
 * t = Gf + rho * ((W - Z) + U) (t = Gf without Z), then
 * W' = kept(group of the entry) ? W - lr * t : +0, every entry kept when mask
 * is NULL.  Each binary32 operation is rounded on its own, in that order. */
void oracle_sgd_step(int64_t A, int64_t B, int64_t C, int64_t D, int32_t kind,
                     const uint8_t *mask, float *W, const float *Gf, const float *Z,
                     const float *U, float rho, float lr)
{
    for (int64_t a = 0; a < A; ++a)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t c = 0; c < C; ++c)
                for (int64_t d = 0; d < D; ++d) {
                    int64_t e = ((a * B + b) * C + c) * D + d;
                    int keep = !mask || mask[group_of(a, b, c, d, B, C, D, kind)];
                    float t = Gf[e];
                    if (Z) {
                        float w_minus_z = W[e] - Z[e];
                        float s = w_minus_z + U[e];
                        float r = rho * s;
                        t = Gf[e] + r;
                    }
                    float q = lr * t;
                    W[e] = keep ? W[e] - q : 0.0f;
                }
}

/* binary32 -> bfloat16 with round to nearest, ties to even, on the 16
 * discarded bits (NaN kept quiet). */
uint16_t oracle_bf16_rne(float x)
{
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t low = u & 0xffffu;
    uint32_t hi = u >> 16;
    if (low > 0x8000u || (low == 0x8000u && (hi & 1u)))
        hi += 1u;
    return (uint16_t)hi;
}

double oracle_bf16_to_double(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

void oracle_bf16_array(int64_t n, const float *x, uint16_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_bf16_rne(x[i]);
}

/* Compaction (Section 3, GEMM lowering with rows / columns removed).
 * For conv group gc the rows are the kept filters a in [gc*A/groups, (gc+1)*A/groups)
 * (row_mask[a], all rows when NULL).  Column (b, c, d) of the group is kept when
 * col_mask[(b*C + c)*D + d], chan_mask[b] and in_ch_mask[gc*B + b] are all set
 * (a NULL mask sets nothing aside).  Columns follow the ascending GEMM column
 * index j = (b*C + c)*D + d, i.e. channel b ascending, then tap.  Each column
 * records col_tap = c*D + d and col_ch = the column's input channel, i.e. the
 * full channel index gc*B + b, or, when in_compacted, its position among the
 * channels with in_ch_mask set (the input then holds only those, ascending).
 * Outputs are concatenated over groups; M_g / K_g get the per-group sizes.
 * Returns 0, or -1 when in_compacted is set without in_ch_mask. */
int oracle_compact(int64_t A, int64_t B, int64_t C, int64_t D, int32_t groups,
                   const float *Z, const uint8_t *row_mask, const uint8_t *col_mask,
                   const uint8_t *chan_mask, const uint8_t *in_ch_mask, int32_t in_compacted,
                   uint16_t *Wc, int32_t *row_idx, int32_t *col_ch, int32_t *col_tap,
                   int32_t *M_g, int32_t *K_g)
{
    if (in_compacted && !in_ch_mask)
        return -1;
    int64_t Ag = A / groups;
    int64_t taps = C * D;
    int64_t wc_off = 0, row_off = 0, col_off = 0;
    int64_t *cb = (int64_t *)malloc(sizeof(int64_t) * (size_t)(B * taps));
    int64_t *ct = (int64_t *)malloc(sizeof(int64_t) * (size_t)(B * taps));
    if (!cb || !ct)
        return -2;
    for (int32_t gc = 0; gc < groups; ++gc) {
        int64_t ncol = 0;
        for (int64_t j = 0; j < B * taps; ++j) {  /* j = b*taps + t: the GEMM column */
            const int64_t b = j / taps;
            const int64_t t = j % taps;
            int keep = 1;
            if (col_mask && !col_mask[j]) keep = 0;
            if (chan_mask && !chan_mask[b]) keep = 0;
            if (in_ch_mask && !in_ch_mask[gc * B + b]) keep = 0;
            if (!keep)
                continue;
            int64_t full = gc * B + b;
            int64_t pos = full;
            if (in_compacted) {
                pos = 0;
                for (int64_t q = 0; q < full; ++q)
                    if (in_ch_mask[q]) ++pos;
            }
            cb[ncol] = b;
            ct[ncol] = t;
            col_ch[col_off + ncol] = (int32_t)pos;
            col_tap[col_off + ncol] = (int32_t)t;
            ++ncol;
        }
        int64_t m = 0;
        for (int64_t a = gc * Ag; a < (gc + 1) * Ag; ++a) {
            if (row_mask && !row_mask[a])
                continue;
            row_idx[row_off + m] = (int32_t)a;
            for (int64_t j = 0; j < ncol; ++j) {
                int64_t c = ct[j] / D, d = ct[j] % D;
                int64_t e = ((a * B + cb[j]) * C + c) * D + d;
                Wc[wc_off + m * ncol + j] = oracle_bf16_rne(Z[e]);
            }
            ++m;
        }
        M_g[gc] = (int32_t)m;
        K_g[gc] = (int32_t)ncol;
        wc_off += m * ncol;
        row_off += m;
        col_off += ncol;
    }
    free(cb);
    free(ct);
    return 0;
}

/* Input preparation: X binary32 NCHW [N, Cin, H, W] -> bfloat16 NCHW [N, Cx, H, W],
 * keeping only the channels with keep[ch] set (all when NULL), ascending. */
void oracle_pack(int64_t N, int64_t Cin, int64_t H, int64_t W, const float *X,
                 const uint8_t *keep, uint16_t *Xb)
{
    int64_t Cx = 0;
    for (int64_t ch = 0; ch < Cin; ++ch)
        if (!keep || keep[ch])
            ++Cx;
    int64_t cx = 0;
    for (int64_t ch = 0; ch < Cin; ++ch) {
        if (keep && !keep[ch])
            continue;
        for (int64_t n = 0; n < N; ++n)
            for (int64_t h = 0; h < H; ++h)
                for (int64_t w = 0; w < W; ++w)
                    Xb[((n * Cx + cx) * H + h) * W + w] =
                        oracle_bf16_rne(X[((n * Cin + ch) * H + h) * W + w]);
        ++cx;
    }
}

/* GEMM-lowered CONV over the compacted matrices (Section 3), by definition:
 * Y[n, p, q, o] = sum_j Wc_g[m, j] * Xb[n, col_ch[j], p*stride - pad + c_j, q*stride - pad + d_j]
 * for output channel o = (rows of earlier groups) + m, (c_j, d_j) = col_tap[j] split
 * by D, zero outside the image, every product and sum in binary64.
 * Xb is bfloat16 NCHW [N, Cx, H, W]; Y is binary64 NHWC [N, P, Q, sum_g M_g]. */
void oracle_conv(int64_t N, int64_t Cx, int64_t H, int64_t W, const uint16_t *Xb,
                 int32_t groups, int64_t C, int64_t D, int64_t stride, int64_t pad,
                 const uint16_t *Wc, const int32_t *M_g, const int32_t *K_g,
                 const int32_t *col_ch, const int32_t *col_tap, double *Y)
{
    int64_t P = (H + 2 * pad - C) / stride + 1;
    int64_t Q = (W + 2 * pad - D) / stride + 1;
    int64_t Cy = 0;
    for (int32_t g = 0; g < groups; ++g)
        Cy += M_g[g];
    /* every output is independent: threads take (image, output row) pairs */
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t p = 0; p < P; ++p) {
            for (int64_t q = 0; q < Q; ++q) {
                int64_t wc_off = 0, col_off = 0, o = 0;
                for (int32_t g = 0; g < groups; ++g) {
                    for (int64_t m = 0; m < M_g[g]; ++m) {
                        double acc = 0.0;
                        for (int64_t j = 0; j < K_g[g]; ++j) {
                            int64_t c = col_tap[col_off + j] / D;
                            int64_t d = col_tap[col_off + j] % D;
                            int64_t h = p * stride - pad + c;
                            int64_t w = q * stride - pad + d;
                            if (h < 0 || h >= H || w < 0 || w >= W)
                                continue;
                            double x = oracle_bf16_to_double(
                                Xb[((n * Cx + col_ch[col_off + j]) * H + h) * W + w]);
                            double wv = oracle_bf16_to_double(Wc[wc_off + m * K_g[g] + j]);
                            acc += wv * x;
                        }
                        Y[((n * P + p) * Q + q) * Cy + o] = acc;
                        ++o;
                    }
                    wc_off += (int64_t)M_g[g] * K_g[g];
                    col_off += K_g[g];
                }
            }
        }
    }
}

/* The non-structured set of Section 3 keeps an arbitrary pattern of weights;
 * the CONV of such a layer is a sparse-matrix product (Section 5 runs it with
 * a CSR sparse library on the GPU).  CSR form of the [A, B*C*D] GEMM matrix:
 * row a lists the columns j with mask[a*B*C*D + j] set, ascending, with values
 * bf16(Z[a*B*C*D + j]) (round to nearest even); row_ptr has A + 1 entries.
 * A kept entry whose value is zero stays an explicit entry.  Returns the
 * number of entries. */
int64_t oracle_csr(int64_t A, int64_t B, int64_t C, int64_t D, const float *Z,
                   const uint8_t *mask, int32_t *row_ptr, int32_t *col, uint16_t *val)
{
    int64_t K = B * C * D, e = 0;
    for (int64_t a = 0; a < A; ++a) {
        row_ptr[a] = (int32_t)e;
        for (int64_t j = 0; j < K; ++j) {
            if (!mask[a * K + j])
                continue;
            col[e] = (int32_t)j;
            val[e] = oracle_bf16_rne(Z[a * K + j]);
            ++e;
        }
    }
    row_ptr[A] = (int32_t)e;
    return e;
}

/* CONV of a CSR layer, by definition: for filter a of conv group
 * gc = a / (A / groups),
 * Y[n, p, q, a] = sum over the entries e of row a of
 *     val[e] * Xb[n, gc*B + b, p*stride - pad + c, q*stride - pad + d],
 * where col[e] = (b*C + c)*D + d; zero outside the image; every product and
 * sum in binary64, entries in row order.  Xb is bfloat16 NCHW
 * [N, groups*B, H, W]; Y is binary64 NHWC [N, P, Q, A]. */
void oracle_conv_csr(int64_t N, int64_t H, int64_t W, const uint16_t *Xb, int64_t A, int64_t B,
                     int64_t C, int64_t D, int32_t groups, int64_t stride, int64_t pad,
                     const int32_t *row_ptr, const int32_t *col, const uint16_t *val, double *Y)
{
    int64_t P = (H + 2 * pad - C) / stride + 1;
    int64_t Q = (W + 2 * pad - D) / stride + 1;
    int64_t Cx = groups * B, per_group = A / groups;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t p = 0; p < P; ++p)
            for (int64_t q = 0; q < Q; ++q)
                for (int64_t a = 0; a < A; ++a) {
                    int64_t gc = a / per_group;
                    double acc = 0.0;
                    for (int64_t e = row_ptr[a]; e < row_ptr[a + 1]; ++e) {
                        int64_t j = col[e];
                        int64_t b = j / (C * D), c = (j / D) % C, d = j % D;
                        int64_t h = p * stride - pad + c;
                        int64_t w = q * stride - pad + d;
                        if (h < 0 || h >= H || w < 0 || w >= W)
                            continue;
                        acc += oracle_bf16_to_double(val[e]) *
                               oracle_bf16_to_double(Xb[((n * Cx + gc * B + b) * H + h) * W + w]);
                    }
                    Y[((n * P + p) * Q + q) * A + a] = acc;
                }
}
