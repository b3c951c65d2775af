/*
 * tvl.h -- C ABI of the TVL GEMV library for AMD Instinct MI355X (gfx950).
 *
 * The operation is the per-token matrix-vector product of a Llama-2 decode
 * step (Kilictas & Alpay, "Bare-Metal Tensor Virtualization", arXiv
 * 2601.03324): Sec. 6.1 defines it by the naive loop y[i] += W[i][j] * x[j]
 * and the GEMV listing "xout = W @ x" with the weight for (i, j) at
 * w + i*n + j; Sec. 1 and Sec. 3.1 state that every token streams every
 * weight matrix once, so the traffic is |W| + |x| + |y| bytes.  Here:
 *
 *     y[i] = sum_{j < K} W[i*ldw + j] * x[j],      0 <= i < M
 *
 *   - W is row-major with a row stride of ldw elements (ldw >= K), fp32 or
 *     binary16 (fp16); x and y are fp32; products are accumulated in fp32.
 *     An fp16 weight is converted to fp32 exactly (subnormals kept).
 *   - Tensor Virtualization Layout (TVL, Sec. 3.2 and the abstract: every
 *     buffer starts on a cache line and every vector load touches one line):
 *     here every row starts on a 128-byte boundary, i.e. W is 128-byte
 *     aligned and ldw * sizeof(weight) is a multiple of 128.  W spans M
 *     whole rows (M * ldw elements, the last row's padding included: a
 *     16-byte load may touch it).  Elements K..ldw-1 of a row are padding;
 *     their values are never used (they may even hold NaN).
 *   - y is overwritten ("xout = W @ x"); its previous contents are ignored.
 *   - Non-finite x: a NaN in x makes every output NaN; an infinite x_j gives
 *     y_i = +-inf by the sign of W_ij, or NaN where W_ij = 0, as IEEE
 *     arithmetic does, in every form whose products are fp32 (all forms but
 *     the fp16 matrix-core form with split x, which is specified for finite
 *     x only; see tvl_item).  With RMSNorm (tvl_item) the normalised x is
 *     NaN at j and 0 elsewhere, so every output is NaN.
 *   - Summation order differs from the sequential loop (Sec. 5.2 accepts the
 *     drift of reordered fused multiply-add accumulation).  Each output is
 *     the sum of 256 interleaved fp32 partial sums (64 lanes x 4) joined by
 *     a fixed tree, so |y_i - exact| <= (K/256 + 8) * 2^-24 * sum_j |W_ij x_j|
 *     up to second-order terms, and reruns of one variant are bitwise equal.
 *
 * Memory and ownership.  All W, x, y pointers are device pointers owned by
 * the caller; the library never allocates, frees or retains them.  The same
 * W or x may appear in several items (a tied classifier, Sec. 5.1; a shared
 * activation).  The library owns only what it allocates itself: plan objects
 * and the K-split workspace (see tvl_gemv), plus one static scratch array per
 * GPU for tvl_gemv_noalloc.
 *
 * Streams.  Every compute call enqueues work on `stream` (0 = the null
 * stream) and returns without synchronising; results are valid once the
 * caller has synchronised with that stream.
 *
 * Errors.  Calls return a tvl_status and never abort or throw.  Arguments are
 * validated before anything is enqueued; a batch with one bad item enqueues
 * nothing.  Launch failures are reported as TVL_ERR_HIP with the HIP error
 * text in tvl_last_error(); faults during execution surface at the caller's
 * next synchronisation, as for any HIP kernel.
 *
 * Threading.  All calls may be made from several host threads.  A plan must
 * not run on two streams at once.  K-split calls that share a stream share
 * one workspace and are ordered by the stream; different streams get
 * different workspaces.
 */
#ifndef TVL_H
#define TVL_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#if defined(__GNUC__)
#define TVL_API __attribute__((visibility("default")))
#else
#define TVL_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

#define TVL_VERSION 100 /* 1.0.0 */

/* Weight element type.  x and y are always fp32.
 *
 * Block-quantised weights (TVL_Q8, TVL_Q4): the paper proposes 4-bit weights
 * unpacked on the fly (Sec. 8.2) and names 4/8-bit quantisation (Sec. 2.2)
 * but fixes no format.  This library's format for an M x K matrix is one
 * 128-byte-aligned buffer:
 *   code plane    M rows of ldw BYTES (ldw a multiple of 128, at least
 *                 roundup(ceil(K*bits/8), 128) = tvl_row_stride);
 *                 8-bit: column j at byte j, two's complement q in [-128, 127];
 *                 4-bit: column j in byte j/2, low nibble first, two's
 *                 complement q in [-8, 7];
 *   scale plane   at byte M*ldw: fp32 in blocks of 4 rows: the scale s_ig
 *                 of columns 64g .. 64g+63 of row i at float index
 *                 (i/4)*4*ng + 4*g + i%4, ng = ceil(K/64), rows padded to
 *                 Mp = M rounded up to a multiple of 4 (entries of rows
 *                 i >= M are padding, never used);
 *   w_ij = s_{i,j/64} * q_ij        (converted exactly; fp32 accumulation;
 *                                    4-bit scales below 2^124: the 4-bit
 *                                    kernels apply 16 s, so larger scales,
 *                                    from weights beyond ~1.5e38, overflow).
 * Keeping the scales out of the code rows keeps every fetched 128-byte line
 * full; the 4-row blocks put the scales of 4 neighbouring rows side by side
 * (one 16-byte load) and the groups of a block in consecutive 16 bytes.  Code bytes past column K are
 * padding and never change the result; the whole buffer spans
 * M*ldw + 4*Mp*ceil(K/64) bytes.  Quantised items take K <= 2^24,
 * ldw <= 2^24 bytes and a scale plane below 2^31 bytes (else TVL_ERR_SHAPE). */
typedef enum tvl_dtype {
    TVL_F32 = 0, /* IEEE binary32 weights */
    TVL_F16 = 1, /* IEEE binary16 weights, converted exactly to fp32 */
    TVL_Q8 = 2,  /* 8-bit block-quantised weights (ldw in bytes) */
    TVL_Q4 = 3   /* 4-bit block-quantised weights (ldw in bytes) */
} tvl_dtype;

typedef enum tvl_status {
    TVL_OK = 0,
    TVL_ERR_NULL = -1,  /* a required pointer is NULL                        */
    TVL_ERR_SHAPE = -2, /* M < 1 or > 2^31-1, K < 1 or > 2^30, ldw < K, ... */
    TVL_ERR_ALIGN = -3, /* W not 128-B aligned, ldw*size % 128 != 0,
                           x not 16-B aligned, y not 4-B aligned             */
    TVL_ERR_DTYPE = -4, /* unknown weight dtype                              */
    TVL_ERR_ALIAS = -5, /* an output overlaps an input or another output     */
    TVL_ERR_HIP = -6,   /* a HIP runtime call or a launch failed             */
    TVL_ERR_NOMEM = -7, /* host or device allocation failed                  */
    TVL_ERR_ARG = -8    /* an unsupported tuning value or other argument     */
} tvl_status;

/* Item operations. */
#define TVL_OP_GEMV 0   /* y = W x                                                */
#define TVL_OP_SWIGLU 1 /* y = silu(W x) * (W3 x), silu(z) = z / (1 + e^-z): the
                           gated FFN input of Sec. 2.1 (W = w1, W3 = w3)          */

/* One GEMV of a batch: y = W x with the same meaning as tvl_gemv's
 * arguments, optionally with its input normalised and/or as a SwiGLU pair,
 * or with several x vectors.  96 bytes, no implicit padding.
 *
 *   RMSNorm (g != NULL; Sec. 2.1 pre-normalisation, Sec. 11.2 listing):
 *     x is replaced by x_j * g_j / sqrt(mean_j(x_j^2) + eps) before the
 *     product.  eps is added to the mean square inside the root, as in the
 *     listing; the root is exact (no reciprocal-root estimate).
 *   SwiGLU (op == TVL_OP_SWIGLU): y_i = silu(a_i) * b_i with a = W x and
 *     b = W3 x over the (normalised) x; W3 has W's M, K, ldw and dtype.
 *   Several vectors (nrhs > 1; beam search with nrhs hypotheses, Sec. 9.1):
 *     y[b*ldy + i] = sum_j W[i*ldw + j] * x[b*ldx + j] for b < nrhs <= 16;
 *     the weights are read once for all vectors.  Only for plain GEMV items
 *     (op == TVL_OP_GEMV, g == NULL).  Up to 4 vectors the products run on
 *     the vector ALUs, from 5 on (by default) on the matrix cores, in fp32
 *     with fp32 accumulation either way; except that launches holding only
 *     fp16 weights use the fp16 matrix cores from 5 vectors on (by default):
 *     each 64- or 128-column chunk of each x vector is scaled by 2^k, which
 *     puts its largest |x| 2^k in [2^13, 2^14), and split into two fp16 parts,
 *     x 2^k = hi + lo + r with |r| <= 2^-22 |x 2^k| + 2^-25; the fp16 products
 *     are exact and accumulate in fp32, and the sum is scaled back exactly.
 *     A chunk in which any nonzero |x 2^k| of any vector is below 2^-7 (a
 *     range wider than the two parts hold) runs on the fp32 matrix cores
 *     instead, so the split adds at most 2^-18 sum_j |W_ij x_j| to the error
 *     bound above, for every finite x.
 *   Block-quantised weights (dtype TVL_Q8 / TVL_Q4): plain one-vector GEMV
 *     items only (op == TVL_OP_GEMV, g == NULL, nrhs <= 1).
 * One launch (plan or batch) may hold plain fp32/fp16 items together with
 * ONE of: RMSNorm/SwiGLU items, several-vector items, quantised items.
 * Items with g != NULL, op != TVL_OP_GEMV or nrhs > 1 run in direct-x mode;
 * they and quantised items cannot be K-split.  Quantised items read x
 * directly too, or, with TVL_FLAG_X_LDS, from a copy of x that each
 * workgroup stages in LDS once per row tile (x of the largest quantised K in
 * the launch, in whole KiB, must fit a workgroup's 160 KB: K <= 40,960;
 * else TVL_ERR_SHAPE); plain items in such a launch still read x directly. */
typedef struct tvl_item {
    const void *W;      /* device, M whole rows of ldw elements of `dtype`   */
    int64_t ldw;        /* row stride in elements                             */
    const float *x;     /* device, K floats                                   */
    float *y;           /* device, M floats, overwritten                      */
    int64_t M;          /* rows                                               */
    int64_t K;          /* columns used                                       */
    int32_t dtype;      /* tvl_dtype                                          */
    int32_t op;         /* TVL_OP_GEMV or TVL_OP_SWIGLU                       */
    const void *W3;     /* TVL_OP_SWIGLU: second matrix (same layout), else NULL */
    const float *g;     /* RMSNorm weight, K floats, 16-byte aligned; NULL = none */
    float eps;          /* RMSNorm epsilon (finite, >= 0; ignored when g == NULL) */
    int32_t nrhs;       /* x vectors: 0 or 1 = one; 2..16 = several           */
    int64_t ldx;        /* nrhs > 1: x row stride in floats (>= K, % 4 == 0)  */
    int64_t ldy;        /* nrhs > 1: y row stride in floats (>= M)            */
} tvl_item;

/* Launch shape override.  A zero field means "choose by shape".
 *   rows_per_wave   R in {1, 2, 4, 8, 16, 32, 64}: rows one wavefront computes
 *                   at once (32 and 64: several-vector launches only)
 *   waves_per_block W in {1, 2, 4, 8}: wavefronts per workgroup
 *   unroll          U in {1, 2, 3, 4, 8}: 16-byte weight loads per row kept in
 *                   flight per lane (several-vector launches: selects the
 *                   matrix-core form, below, where U can exceed 8)
 *   ksplit          S >= 1: K slices per row tile (tvl_gemv only; 1 = row
 *                   split)
 *   grid            workgroups of a sweep launch (0 = one per tile); a smaller
 *                   grid makes each workgroup loop over tiles
 *   flags           TVL_FLAG_X_LDS: stage x once per workgroup in LDS;
 *                   TVL_FLAG_X_DIRECT: each wavefront reads x from global
 *                   memory (L1/L2-cached) next to its weights; neither: the
 *                   library's default mode.
 * Only the triples (R, W, U) the library instantiates for the chosen x mode
 * are accepted (others give TVL_ERR_ARG):
 *   LDS-x:    W=4: (1,4) (1,8) (2,2) (2,3) (2,4) (2,8) (4,1) (4,2) (4,3) (4,4)
 *                  (8,1) (8,2);  W=8: (2,4) (2,8) (4,2);
 *             W=2: (1,8) (2,8) (4,4) (8,2)
 *   direct-x: W=1 and W=4: (1,4) (1,8) (2,2) (2,3) (2,4) (2,8) (4,1) (4,2)
 *                  (4,3) (4,4) (8,1) (8,2);  W=8: (1,8) (2,3) (2,4) (4,2)
 * Launches holding RMSNorm or SwiGLU items (direct-x only):
 *   (2,4,2) (2,4,3) (2,4,4) (2,1,4) (4,1,2) (4,1,4) (4,4,2) (2,1,8) (8,4,1)
 *   (8,2,1) (4,4,3)
 * Launches holding several-vector items (direct-x only), per vector class
 * (nrhs <= 2, <= 4, <= 8) on the vector ALUs:
 *   2: (2,4,2) (2,4,4) (4,4,2) (8,2,1);  8: (2,4,1) (2,4,2) (4,4,1);
 *   4: (2,4,1) (2,4,2) (4,4,1) (4,4,2) (8,4,1) (8,2,1)
 * and, for any nrhs <= 16, on the matrix cores: the 4x4x1 form (rows in
 * groups of 4, U = 1) (8,4,1) (16,1,1) (16,2,1); the 16x16x4 form (rows
 * in groups of 16, U = loads per group in flight) (16,4,8) (32,1,4) (32,2,4)
 * (64,1,4); the 16x16x4 form with rows staged through LDS from registers
 * (U = 2; fp32 and fp16 weights) (16,1,2) (16,4,2) (32,1,2) (32,2,2)
 * (32,4,2) (64,1,2); and the 16x16x4 form with the weights streamed into
 * LDS by the loads themselves (U = 10 S + log2(C / 16) for S LDS stages and
 * chunks of C columns; fp32 and fp16 weights) (16,1,33) (16,2,33) (32,1,33)
 * (16,1,32) (16,4,32) (32,1,32) (32,2,32) (16,4,42) (32,1,42) (32,1,52);
 * and with U + 100 the same for fp16 weights on the fp16 matrix cores with
 * split x (launches holding fp32 weights run the LDS-staged form with the
 * same rows and waves) (16,1,133) (16,2,133) (32,1,133) (32,2,133)
 * (64,1,133) (32,1,132) (64,1,132); and with U = 200 + log2(C / 16) the
 * streamed form with x shared by the block's wavefronts through LDS, fp32 or
 * fp16 weights (launches mixing them run the LDS-staged form with the same
 * rows and waves) (16,4,202) (32,2,202) (32,4,202) (16,2,203) (16,4,203)
 * (16,8,202), and with U + 100 its split-x form for fp16 weights (launches
 * holding fp32 weights run the LDS-staged form) (16,4,303) (32,2,303)
 * (32,4,303) (16,8,303) (16,4,302) (32,4,302), where each wavefront splits
 * x for a quarter (an eighth, a half) of the vectors once per block.  Rows
 * (and, except in the split-x shared form, which reads x through plain
 * pointers, x strides) longer than these forms' buffer descriptors can
 * address (a load's 2, 4 or 8 rows within 2^31 bytes) run the direct-load
 * 16x16x4 form.
 * Launches holding block-quantised items (R rows per group of lanes, see
 * tvl_dtype): direct-x (2,4,2) (4,4,1) (4,4,2) (4,1,2) (8,4,1) (8,2,1);
 * x in LDS (TVL_FLAG_X_LDS; a tuning that sets only the flag keeps the
 * default rows and waves) (4,4,1) (8,4,1) (8,2,1) (4,4,2). */
typedef struct tvl_tuning {
    int32_t rows_per_wave;
    int32_t waves_per_block;
    int32_t unroll;
    int32_t ksplit;
    int32_t grid;
    int32_t flags;
} tvl_tuning;

#define TVL_FLAG_X_LDS 1
#define TVL_FLAG_X_DIRECT 2

/* Opaque sweep plan. */
typedef struct tvl_plan tvl_plan;

/* Library version (TVL_VERSION of the built library). */
TVL_API int32_t tvl_version(void);

/* Row stride, in elements, of the TVL layout for K columns of `dtype`:
 * roundup(K * size, 128) / size; for TVL_Q8 / TVL_Q4 the code row size in
 * bytes, roundup(ceil(K * bits / 8), 128) (see tvl_dtype for the scale
 * plane).  Returns -1 for K < 1 or an unknown dtype.  Pure host function. */
TVL_API int64_t tvl_row_stride(int64_t K, int32_t dtype);

/* TVL pack (Sec. 3.2 alignment): copy a dense row-major [M x K] matrix
 * `src` (device) into `dst` (device, M rows of stride ldw, 128-byte aligned)
 * and zero elements K..ldw-1 of every row.  One kernel launch on `stream`.
 * `src` is only required to be element aligned; `dst` must not overlap `src`.
 * fp32 and fp16 only (quantised rows are written by the quantiser). */
TVL_API tvl_status tvl_pack_rows(void *dst, int64_t ldw, const void *src,
                                 int64_t M, int64_t K, int32_t dtype,
                                 hipStream_t stream);

/* y = W x (Sec. 6.1), one launch.  The library picks the variant by shape
 * (from timings on MI355X): a row split (each wavefront owns R whole rows;
 * one row per single-wavefront workgroup when M is small), or, for very few
 * long rows (M <= 128, rows >= 32 KB), a K split: S workgroups share a row
 * tile, each sums one slice of K into an fp32 partial, and the last
 * workgroup to finish adds the S partials in the fixed order 0..S-1, so
 * results stay deterministic.  The K-split workspace (S*M floats and one
 * counter per row tile) is allocated by the library on first use per
 * (device, stream) and kept until tvl_release_workspaces() or process exit;
 * a first K-split call on a stream that is being captured into a graph
 * fails with TVL_ERR_NOMEM (make one call before capturing).  A workspace
 * replaced by a larger one is not freed either (graphs captured with it
 * stay valid) until tvl_release_workspaces(). */
TVL_API tvl_status tvl_gemv(const void *W, int64_t ldw, int32_t dtype,
                            const float *x, float *y, int64_t M, int64_t K,
                            hipStream_t stream);

/* tvl_gemv with an explicit launch shape (NULL = choose by shape). */
TVL_API tvl_status tvl_gemv_ex(const void *W, int64_t ldw, int32_t dtype,
                               const float *x, float *y, int64_t M, int64_t K,
                               const tvl_tuning *tuning, hipStream_t stream);

/* tvl_gemv_ex for callers that cannot allocate device memory: code that is
 * being captured into a HIP graph, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, same variant choice, same kernels and
 * bitwise the same results as tvl_gemv_ex; it never calls hipMalloc,
 * hipFree or any allocating routine.  Where the variant is a K split, its
 * partials and arrival counters live in a static array of the library
 * (one per GPU, 4.25 MiB, held until the process ends) instead of a
 * per-stream workspace:
 *   - a K split needs S * M <= 2^20 partials and at most 2^16 row tiles
 *     (S: slices, from `tuning` or by shape); larger splits return
 *     TVL_ERR_SHAPE and enqueue nothing.  The default split (M <= 128 rows
 *     of >= 32 KB, S <= 4) always fits;
 *   - every call on one GPU shares that GPU's array, so calls that overlap
 *     on one GPU (concurrent streams or host threads) race and may return
 *     wrong results: order them;
 *   - each launch leaves the counters at zero again; the first call on a
 *     device looks the array up and clears the counters on `stream`, then
 *     synchronises `stream`.  That first call must not be captured: while
 *     `stream` is capturing it returns TVL_ERR_ARG and enqueues nothing.
 *     Later calls make no HIP call besides the launch. */
TVL_API tvl_status tvl_gemv_noalloc(const void *W, int64_t ldw, int32_t dtype,
                                    const float *x, float *y, int64_t M, int64_t K,
                                    const tvl_tuning *tuning, hipStream_t stream);

/* One item (any op, with or without RMSNorm) in one launch.  A plain GEMV
 * item is the same as tvl_gemv_ex; fused items use the direct-x row split.
 * `tuning` may be NULL. */
TVL_API tvl_status tvl_gemv_item(const tvl_item *item, const tvl_tuning *tuning,
                                 hipStream_t stream);

/* All n GEMVs of `items` (e.g. every weight matrix of one decode token,
 * Sec. 1: each token streams every matrix once) in ONE launch.  The host
 * array `items` is read during the call only.  The first call with a given
 * item list builds a device tile table (one synchronous upload) and caches
 * it; later calls with an identical list launch at once.  The cache holds 64
 * lists; when it is full the device is synchronised and the cache emptied.
 * While `stream` is being captured into a graph, only a list that already
 * has a cached plan launches (any other returns TVL_ERR_ARG and enqueues
 * nothing: building a plan allocates and uploads); a plan launched into a
 * capture is kept past eviction, until tvl_release_workspaces().
 * No output y may overlap any W, x or other y of the batch. */
TVL_API tvl_status tvl_gemv_batch_sweep(const tvl_item *items, int32_t n,
                                        hipStream_t stream);

/* Sweep plan: validate `items`, build the tile table (tiles of R*W output
 * rows; R/2*W for SwiGLU items; R*W*64/G for quantised items whose rows use
 * G lanes each; ordered by bytes per tile, largest first; in plans with
 * several-vector or quantised items, each item's tiles are kept on as few
 * of the GPU's XCDs as the largest-first order allows, so each XCD's L2
 * fetches fewer x vectors) and upload it once.  The item
 * list is copied; the W, x, y buffers it names must stay valid for every
 * run.  `tuning` may be NULL.  The plan belongs to the device current at
 * creation.  Not while a stream of that device is being captured (the table
 * is uploaded synchronously); running a plan may be captured. */
TVL_API tvl_status tvl_sweep_plan_create(const tvl_item *items, int32_t n,
                                         const tvl_tuning *tuning,
                                         tvl_plan **plan);
/* Run a plan: exactly one kernel launch on `stream` (none for a plan of no
 * items). */
TVL_API tvl_status tvl_sweep_plan_run(const tvl_plan *plan, hipStream_t stream);
/* Number of tiles and the launch grid of a plan (either pointer may be NULL). */
TVL_API tvl_status tvl_sweep_plan_info(const tvl_plan *plan, int64_t *ntiles,
                                       int64_t *grid, int32_t *rows_per_tile);
/* Free a plan (synchronises its device first).  NULL is a no-op.  Graphs
 * that captured a run of the plan must not be replayed afterwards. */
TVL_API tvl_status tvl_sweep_plan_destroy(tvl_plan *plan);

/* Free the K-split workspaces and the batch-sweep cache, including those
 * kept for captured graphs (synchronises every device that holds one).
 * Graphs that captured K-split or tvl_gemv_batch_sweep calls must not be
 * replayed afterwards. */
TVL_API tvl_status tvl_release_workspaces(void);

/* Diagnostics (not part of the GEMV path; used to calibrate measurements).
 * tvl_util_read_stream: read `bytes` (a multiple of 16) at `src` (16-byte
 *   aligned) with the same streaming loads as the GEMV, in `sink_len`
 *   workgroups each reading one contiguous span, and write one float per
 *   workgroup to `sink` (`sink_len` floats; the sum read by its first
 *   thread).  *grid_out (may be NULL) receives the grid, which equals
 *   sink_len.
 * tvl_util_copy: copy `bytes` (multiple of 16, both 16-byte aligned, no
 *   overlap) from src to dst. */
TVL_API tvl_status tvl_util_read_stream(const void *src, int64_t bytes,
                                        float *sink, int64_t sink_len,
                                        int64_t *grid_out, hipStream_t stream);
TVL_API tvl_status tvl_util_copy(void *dst, const void *src, int64_t bytes,
                                 hipStream_t stream);

/* Static text for a status code. */
TVL_API const char *tvl_status_str(int32_t status);
/* Detail of the last failure on the calling thread ("" if none). */
TVL_API const char *tvl_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TVL_H */
