/*
 * structadmm.h -- C ABI of the MI355X (gfx950) StructADMM hot path.
 *
 * Method: "StructADMM: A Systematic, High-Efficiency Framework of Structured
 * Weight Pruning for DNNs" (arXiv 1807.11091).
 *
 * The library computes, on one GPU:
 *   - the Z-update of the ADMM regularisation step (Section 4, eq. (4) and
 *     "Solving the second subproblem"): Z = Euclidean projection of W + U
 *     onto a filter-, channel-, filter-shape-wise or non-structured sparsity
 *     set (Section 3), fused optionally with the dual update
 *     U <- U + W - Z (Section 4, below eq. (3)) and the gradient of the
 *     quadratic term of eq. (3), G = rho * (W - Z + U);
 *   - the standalone dual update / gradient;
 *   - one SGD step of the W-subproblem or of masked retraining (Section 4);
 *   - the compaction of a pruned layer into the smaller dense GEMM matrix
 *     that filter (row) and channel / shape (column) pruning leave
 *     (Section 3, "Combination of structured sparsities");
 *   - the CONV over that compacted matrix as an implicit GEMM on the bf16
 *     matrix cores (the same kernel with an uncompacted matrix is the dense
 *     baseline);
 *   - for non-structured (element-wise) pruning, the CSR form of the layer
 *     and its CONV as a sparse product (Section 5's comparison).
 *
 * Conventions shared by every entry point
 *   - Every tensor argument is DEVICE memory owned by the caller.  The
 *     library never allocates or frees device memory; scratch space comes
 *     from the caller (see structadmm_project_workspace).
 *   - Weights are binary32, contiguous, in [A, B, C, D] order (filters,
 *     channels per conv group, kernel height, kernel width), i.e. PyTorch /
 *     Caffe OIHW.  The flat index of (a, b, c, d) is ((a*B + b)*C + c)*D + d
 *     and the GEMM column of (b, c, d) is j = (b*C + c)*D + d.
 *   - Work is enqueued asynchronously on the given HIP stream (0 = the null
 *     stream).  Only structadmm_compact and structadmm_compact_many synchronise with the host.
 *   - Return value 0 = success; negative = error (codes below).  All
 *     arguments are validated on the host before anything is enqueued, so
 *     an error return leaves every output untouched.
 *     structadmm_last_error() gives a message for the calling thread.
 *   - Identical inputs give bitwise identical outputs (no floating-point
 *     atomics; every reduction has a fixed order).
 *   - Calls on different streams over disjoint buffers may overlap; calls
 *     that share output buffers must be ordered by the caller.
 */
#ifndef STRUCTADMM_H
#define STRUCTADMM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- error codes ---------------------------------------------------- */
#define SA_OK 0
#define SA_E_ARG (-1)         /* null required pointer, bad size, k out of range, ... */
#define SA_E_ALIGN (-2)       /* a pointer lacks the alignment stated below */
#define SA_E_WORKSPACE (-3)   /* workspace missing or smaller than the size query */
#define SA_E_UNSUPPORTED (-4) /* valid request outside what the kernels implement */
#define SA_E_HIP (-5)         /* a HIP runtime call or kernel launch failed */

/* ---- constraint sets (Section 3) ------------------------------------ */
typedef enum {
    SA_FILTER = 0,  /* at most k nonzero filters  X[a,:,:,:]; n_groups = A        */
    SA_CHANNEL = 1, /* at most k nonzero channels X[:,b,:,:]; n_groups = B        */
    SA_SHAPE = 2,   /* at most k nonzero vectors  X[:,b,c,d]; n_groups = B*C*D    */
    SA_ELEMENT = 3  /* at most k nonzero weights;             n_groups = A*B*C*D  */
} sa_kind;

/* Largest group count the structured selection handles (filter / channel /
 * shape).  The element-wise selection has no such limit (n < 2^31). */
#define SA_MAX_STRUCT_GROUPS 8192
/* Largest number of conv groups of a layer. */
#define SA_MAX_CONV_GROUPS 16

/* ---- Z-update: structadmm_project ----------------------------------- */
/*
 * One layer of the Z-update (Section 4).  With V = fl32(W + U) (one binary32
 * add per entry):
 *   score of group g: O_g = sum over the group of (double)v * (double)v
 *     (squared Frobenius norm, binary64 accumulation); element-wise: |v|;
 *   the k groups with the largest scores are kept, exactly k of them; ties
 *     at the k-th score go to the lowest group index;
 *   Z = v on kept groups, +0 elsewhere.
 * Fused step (G != NULL): with the same W, U' = fl32(v - Z) is written to U
 *   (the dual update U + W - Z) and G = fl32(rho * fl32(fl32(W - Z) + U'))
 *   (the gradient of rho/2 ||W - Z + U'||^2, eq. (3)).
 * in_ch_mask (optional): a fixed input-channel support.  Entry gc*B + b
 *   (conv group gc = a / (A/groups)) set to 0 forces Z to 0 on the slice
 *   X[a in group gc, b, :, :]; those entries do not enter any score, so the
 *   result is the projection onto the intersection of the two sets.
 *   Supported with every kind.  When in_ch_mask aliases the mask output of an
 *   earlier layer of the same call (same pointer), that layer is completed
 *   first: layers are processed in array order of such dependencies.
 */
typedef struct sa_project_desc {
    int64_t A, B, C, D;        /* weight tensor shape, each >= 1; A*B*C*D < 2^31 */
    int32_t groups;            /* conv groups, >= 1, A % groups == 0            */
    int32_t kind;              /* sa_kind                                       */
    int64_t k;                 /* kept groups, 0 <= k <= n_groups               */
    const float *W;            /* [A,B,C,D] binary32, 16-byte aligned            */
    float *U;                  /* [A,B,C,D] binary32, 16-byte aligned; read, and
                                  overwritten with U' when G != NULL            */
    const uint8_t *in_ch_mask; /* [groups*B] or NULL                            */
    float *Z;                  /* out [A,B,C,D], 16-byte aligned; must not alias W or U */
    uint8_t *mask;             /* out [n_groups]: 1 = kept, 0 = pruned          */
    int32_t *kept_idx;         /* out [k]: kept group indices, ascending (may be NULL when k == 0) */
    double *scores;            /* out [n_groups] scores, or NULL                */
    float rho;                 /* penalty rho of eq. (3) (fused step only)      */
    float *G;                  /* out [A,B,C,D], 16-byte aligned, or NULL (no fused step) */
} sa_project_desc;

/* Workspace bytes that structadmm_project needs for these layers (0 if none).
 * Returns 0 also for invalid descriptors; structadmm_project reports those. */
size_t structadmm_project_workspace(const sa_project_desc *layers, int n_layers);

/* Z-update (and optional fused dual update + gradient) of n_layers layers.
 * ws: device workspace of at least structadmm_project_workspace() bytes,
 * 256-byte aligned, reused freely by the library during the call's kernels
 * (calls sharing one workspace must be ordered). */
int structadmm_project(const sa_project_desc *layers, int n_layers, void *ws, size_t ws_bytes,
                       hipStream_t stream);

/* Largest scratch structadmm_project_noalloc can use (bytes). */
#define SA_PROJECT_NOALLOC_BYTES (16u << 20)

/* structadmm_project without a caller workspace and without any device
 * allocation: for callers that cannot allocate (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  Same layers, same
 * results as structadmm_project; its scratch is a fixed array of
 * SA_PROJECT_NOALLOC_BYTES held by the library on each GPU it runs on (the
 * GPU current at the call) until the process ends.  Returns SA_E_WORKSPACE,
 * before anything is enqueued, when the layers need more scratch than that
 * (structadmm_project_workspace() > SA_PROJECT_NOALLOC_BYTES).  Every call on
 * one GPU shares that GPU's array: calls that may overlap on one GPU (other
 * streams, other threads) race and must be ordered by the caller. */
int structadmm_project_noalloc(const sa_project_desc *layers, int n_layers, hipStream_t stream);

/* ---- dual update / gradient: structadmm_dual_update ------------------ */
/*
 * U <- fl32(fl32(U + W) - Z) (Section 4, below eq. (3)) when update_dual != 0,
 * and G = fl32(rho * fl32(fl32(W - Z) + U)) with the (new) U: the gradient of
 * rho/2 ||W - Z + U||_F^2 (eq. (3)) that each SGD step of the W-subproblem adds.
 * G may be NULL (dual update only).  All arrays binary32 [n], 16-byte aligned.
 */
typedef struct sa_dual_desc {
    int64_t n;          /* entries, 1 <= n < 2^31 */
    const float *W;
    const float *Z;
    float *U;           /* in/out */
    float rho;
    float *G;           /* out or NULL */
    int32_t update_dual;
} sa_dual_desc;

int structadmm_dual_update(const sa_dual_desc *layers, int n_layers, hipStream_t stream);

/* ---- W-subproblem SGD step / masked retraining: structadmm_sgd_step -- */
/*
 * One stochastic-gradient step on a layer's weights (Section 4).  During ADMM
 * regularisation the W-subproblem (eq. (3)) adds rho/2 ||W - Z + U||_F^2 to the
 * loss; in masked retraining ("Masked mapping and retraining") the weights of
 * pruned groups are held at zero while the rest train on.
 *   t  = Gf + rho * ((W - Z) + U)          (t = Gf when Z is NULL)
 *   W' = keep(group of e) ? W - lr * t : +0  (every entry kept when mask is NULL)
 * in binary32, each operation rounded in this order: d = W - Z, s = d + U,
 * r = rho * s, t = Gf + r, q = lr * t, W' = W - q.  Gf is the loss gradient from
 * the caller's backward pass.  mask is a group mask as structadmm_project writes
 * it for (A, B, C, D, kind): group of entry (a, b, c, d) = a (filter), b
 * (channel), (b*C + c)*D + d (shape), the entry itself (element).
 * W is updated in place.  Float arrays: [A,B,C,D] binary32, 16-byte aligned;
 * Z and U are both given or both NULL; Gf may not alias W.
 */
typedef struct sa_sgd_desc {
    int64_t A, B, C, D;      /* shape; A*B*C*D < 2^31 */
    int32_t kind;            /* group map of mask: SA_FILTER .. SA_ELEMENT */
    const uint8_t *mask;     /* [n_groups] (1 = kept) or NULL */
    float *W;                /* in/out */
    const float *Gf;         /* loss gradient */
    const float *Z;          /* NULL: no ADMM term */
    const float *U;          /* NULL exactly when Z is NULL */
    float rho;
    float lr;
} sa_sgd_desc;

int structadmm_sgd_step(const sa_sgd_desc *layers, int n_layers, hipStream_t stream);

/* ---- compaction: structadmm_compact --------------------------------- */
/*
 * Builds, per conv group gc, the dense GEMM matrix that remains after row and
 * column pruning (Section 3):
 *   rows: the filters a in [gc*A/groups, (gc+1)*A/groups) with row_mask[a] set
 *         (every row when row_mask is NULL), ascending;
 *   columns: the pairs (tap t = c*D + d, channel b) with col_mask[b*C*D + t],
 *         chan_mask[b] and in_ch_mask[gc*B + b] all set (a NULL mask sets
 *         nothing aside).  When col_mask is NULL and the kept channels sit at
 *         consecutive input positions (sizes->run > 0), in tap-major order:
 *         t ascending, then b ascending; otherwise in channel-major order:
 *         b ascending, then t ascending;
 *   entries: Wc[m][j] = Z[row m, column j] rounded to bfloat16 (nearest even).
 * Matrices are concatenated over conv groups, each row-major [M_g][ldk_g]
 * with ldk_g = K_g rounded up to a multiple of 64; the padding columns
 * j in [K_g, ldk_g) hold +0 (rows start 128-byte aligned and the CONV reads
 * whole 64-column slices without a bounds check).
 * Column tables: col_tap[j] = c*D + d, col_ch[j] = input channel of column j,
 * i.e. gc*B + b, or, when in_compacted is set, the position of channel
 * gc*B + b among the channels with in_ch_mask set (the input then holds only
 * those channels, ascending).  row_idx lists the kept filters (the output
 * channel order of structadmm_conv_fwd).
 * Alignment columns: when the input is channel-compacted to a multiple of 8
 * channels and a group keeps every tap of one run of consecutive input
 * positions that does not start and end on a multiple of 8, the group's
 * columns are widened to the enclosing 8-aligned window of positions when it
 * is at most 1.5 times the run: the window's other positions (channels of a
 * neighbouring group) become columns whose entries are +0 (kpad counts them),
 * so the run is whole 16-byte vectors of every pixel and the CONV takes its
 * direct kernels.  Their products are +0 for finite inputs, so the CONV's
 * result is that of the kept columns alone.
 * Masks are byte arrays (0 = pruned) such as structadmm_project's mask.
 * Synchronises with the host and fills *sizes.
 */
typedef struct sa_compact_desc {
    int64_t A, B, C, D;          /* shape of Z */
    int32_t groups;              /* 1 <= groups <= SA_MAX_CONV_GROUPS, A % groups == 0 */
    const float *Z;              /* [A,B,C,D] binary32 */
    const uint8_t *row_mask;     /* [A] or NULL            */
    const uint8_t *col_mask;     /* [B*C*D] or NULL        */
    const uint8_t *chan_mask;    /* [B] or NULL            */
    const uint8_t *in_ch_mask;   /* [groups*B] or NULL     */
    int32_t in_compacted;        /* requires in_ch_mask    */
    uint16_t *Wc;                /* out, capacity A * roundup(B*C*D, 64) bfloat16 */
    int32_t *row_idx;            /* out, capacity A                     */
    int32_t *col_ch;             /* out, capacity groups*B*C*D          */
    int32_t *col_tap;            /* out, capacity groups*B*C*D          */
    void *ws;                    /* device scratch, >= SA_COMPACT_WS_BYTES, 256-byte aligned */
} sa_compact_desc;

#define SA_COMPACT_WS_BYTES 4096

typedef struct sa_compact_sizes {
    int32_t groups;
    int32_t M[SA_MAX_CONV_GROUPS];          /* kept rows of each conv group     */
    int32_t K[SA_MAX_CONV_GROUPS];          /* kept columns of each conv group  */
    int32_t ldk[SA_MAX_CONV_GROUPS];        /* row stride of group gc in Wc     */
    int64_t wc_offset[SA_MAX_CONV_GROUPS];  /* element offset of group gc in Wc */
    int32_t row_offset[SA_MAX_CONV_GROUPS]; /* offset in row_idx / output channels */
    int32_t col_offset[SA_MAX_CONV_GROUPS]; /* offset in col_ch / col_tap       */
    /* run[gc] > 0 when the group's columns are every tap times one run of
     * run[gc] consecutive input channels starting at run_base[gc] (a dense
     * channel block: filter / channel pruning); 0 for a general gather. */
    int32_t run[SA_MAX_CONV_GROUPS];
    int32_t run_base[SA_MAX_CONV_GROUPS];
    /* Input channels the group's columns read lie in [ch_lo[gc], ch_lo[gc] + ch_span[gc])
     * (ch_span = 0 when the group has no column). */
    int32_t ch_lo[SA_MAX_CONV_GROUPS];
    int32_t ch_span[SA_MAX_CONV_GROUPS];
    /* Of the K[gc] columns, the number added for alignment (see below); the
     * kept columns are K[gc] - kpad[gc]. */
    int32_t kpad[SA_MAX_CONV_GROUPS];
} sa_compact_sizes;

int structadmm_compact(const sa_compact_desc *desc, sa_compact_sizes *sizes, hipStream_t stream);

/* The compactions of n descriptors (the layers of a network after one
 * projection, Section 3) with one wait of the host: the kernels of every
 * descriptor are enqueued, then the host waits once for all the sizes
 * (twice when a descriptor has in_compacted set).  Results are those of n
 * calls of structadmm_compact; sizes[i] belongs to descs[i].  Every
 * descriptor needs its own ws (scratch ranges of SA_COMPACT_WS_BYTES may not
 * overlap: SA_E_ARG) and outputs that no other descriptor writes.  All
 * descriptors are validated before anything is enqueued, so an error leaves
 * every output untouched.  n = 0 does nothing. */
int structadmm_compact_many(const sa_compact_desc *descs, int32_t n, sa_compact_sizes *sizes, hipStream_t stream);

/* ---- input layout: structadmm_pack_nhwc ------------------------------ */
/*
 * X binary32 NCHW [N, Cin, H, W] -> Xp bfloat16 NHWC [N, H, W, Cx] (round to
 * nearest even), keeping the channels with keep[ch] set (all when NULL) in
 * ascending order; Cx must equal the number of kept channels.
 */
int structadmm_pack_nhwc(const float *X, int32_t N, int32_t Cin, int32_t H, int32_t W,
                         const uint8_t *keep, int32_t Cx, uint16_t *Xp, hipStream_t stream);

/* ---- compacted CONV: structadmm_conv_fwd ----------------------------- */
/*
 * Section 3, "Combination of structured sparsities": the CONV lowered to a GEMM
 * over the compacted weight matrix.  Pruning removes rows (filters) or
 * columns (channels, filter shapes) of the [A, B*C*D] matrix; what remains is
 * a smaller full GEMM with the same products and sums as the dense CONV with
 * the pruned weights set to zero, on the kept output channels:
 * Y[n, p, q, o] = sum_j Wc_g[m, j] * X[n, p*stride - pad + c_j, q*stride - pad + d_j, col_ch[j]]
 * for conv group g, output channel o = sizes->row_offset[g] + m, (c_j, d_j) =
 * (col_tap[j] / D, col_tap[j] % D); zero outside the image (cross-correlation,
 * no bias, no dilation).  bfloat16 inputs, binary32 accumulation on the
 * matrix cores, bfloat16 output (nearest even).
 * X: bfloat16 NHWC [N, H, W, Cx], 16-byte aligned, smaller than 2 GiB.
 * Y: bfloat16 NHWC [N, P, Q, Cy], Cy = sum_g M_g, P = (H + 2*pad - C)/stride + 1,
 * same for Q, 4-byte aligned; with ldy > 0 its N*P*Q rows are ldy >= Cy
 * elements apart instead of Cy (a padded channel pitch: with ldy a multiple
 * of 8 every row starts on a 16-byte boundary, so the output is written with
 * 16-byte stores when Cy is not a multiple of 8).  Elements [Cy, ldy) of a row
 * are not part of the result: the call leaves them unchanged or writes +0
 * there.
 * sizes: host struct filled by structadmm_compact for the same Wc / tables.
 */
typedef struct sa_conv_desc {
    int32_t N, H, W, Cx;         /* input */
    int32_t C, D;                /* kernel height, width */
    int32_t stride, pad;
    const sa_compact_sizes *sizes; /* host pointer */
    const uint16_t *X;
    const uint16_t *Wc;
    const int32_t *col_ch;
    const int32_t *col_tap;
    uint16_t *Y;
    void *ws;                    /* device scratch of structadmm_conv_workspace() bytes,
                                    256-byte aligned (NULL when that size is 0) */
    size_t ws_bytes;
    int32_t ldy;                 /* output row pitch in elements (0: Cy) */
} sa_conv_desc;

/* Scratch bytes structadmm_conv_fwd needs.  None when the input has a
 * multiple of 8 channels and each group's input footprint fits in LDS (any
 * column set).  An input with other channel counts is first rewritten as its
 * space-to-depth image (bfloat16, channels padded to a multiple of 8) in the
 * scratch; a group whose footprint does not fit in LDS first gathers its
 * compacted im2col rows, N*P*Q x ldk bfloat16, into a region of its own.
 * Returns 0 for an invalid descriptor; structadmm_conv_fwd reports those. */
size_t structadmm_conv_workspace(const sa_conv_desc *desc);

/* Asynchronous on `stream`.  Returns SA_OK, or a negative code with the
 * thread's message set (nothing enqueued): SA_E_ARG for shapes, sizes or
 * pointers that do not fit the descriptor, SA_E_ALIGN for misaligned X / Y /
 * scratch, SA_E_WORKSPACE when ws is smaller than structadmm_conv_workspace(),
 * SA_E_UNSUPPORTED beyond the limits above, SA_E_HIP for a failed launch. */
int structadmm_conv_fwd(const sa_conv_desc *desc, hipStream_t stream);

/* Which kernels structadmm_conv_fwd takes for a descriptor (Section 3: the
 * compacted CONV is a GEMM over the kept rows and columns; the library picks
 * a kernel per conv group from the column set and the sizes).  Host only: no
 * GPU work, the device pointers are not read.  Same validation and error
 * codes as structadmm_conv_fwd; on success *info is filled. */
#define SA_CONV_NONE 0       /* group without output channels                          */
#define SA_CONV_DIRECT 1     /* every tap of a channel run, LDS-staged 64/128-filter tiles  */
#define SA_CONV_DIRECT_IG 2  /* every tap of a channel run, 16-filter-granular tiles       */
#define SA_CONV_FOOTPRINT 3  /* any columns, input footprint of the pixel tile in LDS      */
#define SA_CONV_GATHER 4     /* any columns, im2col rows gathered to scratch first         */
typedef struct sa_conv_plan_info {
    int32_t groups;
    int32_t path[SA_MAX_CONV_GROUPS]; /* SA_CONV_* per conv group                         */
    int32_t ksplit;                   /* > 1: columns split over workgroups (small batch) */
    int32_t space_to_depth;           /* stride of the space-to-depth image, 0 = none     */
    int32_t ig_tile[4];               /* SA_CONV_DIRECT_IG: MT, NF, WM = 16*MT*WM filters by
                                         64*NF/WM pixels per tile, and 1 (every tile
                                         runs whole in one workgroup of four wavefronts)  */
    int32_t footprint_tile[3];        /* SA_CONV_FOOTPRINT: TM, TN, NW = 32*TM filters by
                                         32*NW*TN pixels per workgroup                    */
} sa_conv_plan_info;
int structadmm_conv_plan(const sa_conv_desc *desc, sa_conv_plan_info *info);

/* ---- non-structured layers as CSR: structadmm_csr -------------------- */
/*
 * The non-structured set of Section 3 keeps an arbitrary pattern of weights,
 * which leaves no smaller dense GEMM; its CONV is a sparse-matrix product
 * (Section 5 runs it with a CSR sparse library and finds little or no
 * speedup).  From the ascending kept indices of an element-wise projection
 * (structadmm_project with kind SA_ELEMENT: flat indices a*B*C*D + j), builds
 * the CSR form of the [A, B*C*D] GEMM matrix:
 *   row_ptr[a] = number of kept indices below a*B*C*D (row_ptr[A] = nnz),
 *   col[e]     = kept_idx[e] - a*B*C*D for row_ptr[a] <= e < row_ptr[a+1],
 *   val[e]     = bfloat16(Z[kept_idx[e]]) (round to nearest even).
 * kept_idx must be strictly ascending and below A*B*C*D (as the projection
 * writes it); it is not re-validated on the device, where an index out of
 * range yields a zero entry instead of an out-of-bounds access.
 */
typedef struct sa_csr_desc {
    int64_t A, B, C, D;        /* weight tensor shape; A*B*C*D < 2^31           */
    int64_t nnz;               /* number of kept weights, 0 <= nnz <= A*B*C*D  */
    const float *Z;            /* [A,B,C,D] binary32                            */
    const int32_t *kept_idx;   /* [nnz] ascending flat indices (NULL if nnz == 0) */
    int32_t *row_ptr;          /* out [A+1]                                     */
    int32_t *col;              /* out [nnz] (NULL if nnz == 0)                  */
    uint16_t *val;             /* out [nnz] bfloat16 bits (NULL if nnz == 0)   */
} sa_csr_desc;

int structadmm_csr(const sa_csr_desc *desc, hipStream_t stream);

/* ---- sparse CONV of a CSR layer: structadmm_conv_sparse_fwd ---------- */
/*
 * Y[n, p, q, a] = sum over the entries e of row a of
 *     val[e] * X[n, p*stride - pad + c, q*stride - pad + d, gc*B + b]
 * with conv group gc = a / (A / groups) and col[e] = (b*C + c)*D + d; zero
 * outside the image (cross-correlation, no bias, no dilation).  bfloat16
 * operands, binary32 accumulation (packed bf16 dot products on the vector
 * ALUs: a pattern of single weights has no dense tile for the matrix cores),
 * bfloat16 output (nearest even).  The result equals structadmm_conv_fwd over
 * the uncompacted matrix of the same weights up to the order of the sums.
 * X: bfloat16 NHWC [N, H, W, Cx], Cx = groups*B a multiple of 8, 16-byte
 *    aligned, smaller than 2 GiB.
 * Y: bfloat16 NHWC [N, P, Q, A], P = (H + 2*pad - C)/stride + 1, same for Q,
 *    16-byte aligned.
 * The input footprint of a tile of output pixels (the conv group's channels)
 * must fit in LDS (SA_E_UNSUPPORTED otherwise).
 */
typedef struct sa_sparse_conv_desc {
    int32_t N, H, W, Cx;       /* input */
    int32_t A, B, C, D;        /* weight tensor shape */
    int32_t groups, stride, pad;
    int64_t nnz;               /* row_ptr[A] */
    const uint16_t *X;
    const int32_t *row_ptr;    /* [A+1], as structadmm_csr writes it */
    const int32_t *col;        /* [nnz] */
    const uint16_t *val;       /* [nnz] bfloat16 bits */
    uint16_t *Y;
    void *ws;                  /* device scratch of structadmm_conv_sparse_workspace()
                                  bytes, 256-byte aligned: the entries' LDS offsets
                                  and values with every row padded to 8 entries */
    size_t ws_bytes;
    int32_t reuse_ws;          /* 0: (re)build the padded entries in ws, then run
                                  the CONV.  Nonzero: ws already holds what an
                                  earlier call with the same row_ptr, col, val,
                                  nnz, shape, groups and geometry (N, H, W, Cx,
                                  stride, pad) built, and only the CONV runs (a
                                  layer's CSR is fixed once it is pruned) */
} sa_sparse_conv_desc;

/* Scratch bytes structadmm_conv_sparse_fwd needs (0 for an invalid descriptor). */
size_t structadmm_conv_sparse_workspace(const sa_sparse_conv_desc *desc);

int structadmm_conv_sparse_fwd(const sa_sparse_conv_desc *desc, hipStream_t stream);

/* Message describing the last error on the calling thread ("" if none). */
const char *structadmm_last_error(void);

/* Library version string. */
const char *structadmm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* STRUCTADMM_H */
