/*
 * libbsr -- block-sparse-row (BSR) weights times dense activations on AMD MI355X (gfx950).
 *
 * The operations are those of "Algorithm to Compilation Co-design: An Integrated View of Neural
 * Network Sparsity" (Guo & Huang, 2021):
 *   - block-magnitude pruning of a dense weight (Sec. 2.1, Eq. 2 and Eq. 3): partition W into
 *     R x C blocks, score each block by its l2 norm, keep the k blocks with the largest norm;
 *   - the BSR storage of the pruned weight as data, indices and indptr in SciPy's layout
 *     (Sec. 2.2, second bullet);
 *   - the sparse-weight x dense-input product that touches only stored blocks (Sec. 2.2, first and
 *     second bullets), applied to the BERT attention projections (Sec. 2.3): Y = X W^T + b.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Shapes.  W is N x K, row-major, laid out [out][in] like a linear layer's weight.  A block shape
 *   R x C means R output rows by C input columns; R must divide N and C must divide K.  Then
 *   Nb = N / R block-rows, Kb = K / C block-columns, nb = Nb * Kb blocks.  Block (i, j) covers
 *   W[iR:(i+1)R, jC:(j+1)C] and has the row-major id i * Kb + j.
 * BSR layout.  indptr int32[Nb + 1] with indptr[0] = 0, non-decreasing, indptr[Nb] = nnzb;
 *   indices int32[nnzb], strictly ascending inside each block-row, each < Kb;
 *   data [nnzb][R][C] row-major (fp32, or bf16 as raw uint16 bit patterns).
 * Activations.  X is T x K row-major with row pitch ldx >= K elements (T = batch * sequence);
 *   Y is T x N fp32 row-major with row pitch ldy >= N.  Bias is fp32[N] or NULL (adds +0).
 * Memory.  Every data pointer is a device pointer (hipMalloc or torch memory) owned by the
 *   caller.  The library never allocates, frees or synchronises; it only enqueues kernels.
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = the null stream).  All work is
 *   stream-ordered; results are visible after the caller synchronises that stream.
 * Errors.  Arguments are validated on the host before anything is enqueued; on error nothing is
 *   launched and outputs are untouched.  A launch failure reported by the HIP runtime returns
 *   BSR_ERR_HIP.  Device contents (indptr, indices) cannot be checked without a synchronisation,
 *   so they are trusted; kernels clamp every index they read to the declared array bounds, so a
 *   malformed matrix yields wrong values but no out-of-bounds access.
 * Concurrency.  A bsr_matrix_t is read-only to the library and may be used on several streams at
 *   once.  X, Y, W and workspaces must not overlap each other.
 */
#ifndef LIBBSR_H
#define LIBBSR_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define LIBBSR_API __attribute__((visibility("default")))
#else
#define LIBBSR_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BSR_OK = 0,
    BSR_ERR_NULL = 1,       /* a required pointer is NULL                                      */
    BSR_ERR_SHAPE = 2,      /* R does not divide N, C does not divide K, ld < width, T < 0      */
    BSR_ERR_ARG = 3,        /* density NaN or outside [0, 1]; k outside [0, nb]; bad dtype enum */
    BSR_ERR_DTYPE = 4,      /* X dtype differs from the BSR data dtype                          */
    BSR_ERR_CAPACITY = 5,   /* output arrays too small for k blocks                             */
    BSR_ERR_WORKSPACE = 6,  /* workspace NULL or smaller than bsr_prune_workspace_bytes()       */
    BSR_ERR_HIP = 7,        /* the HIP runtime reported an error                                */
    BSR_ERR_ARCH = 8,       /* the current device is not gfx950                                 */
    BSR_ERR_UNSUPPORTED = 9 /* valid arguments outside what the library implements (e.g. sizes
                               beyond int32 element offsets)                                    */
} bsr_status;

typedef enum { BSR_F32 = 0, BSR_BF16 = 1 } bsr_dtype;

/* A BSR matrix in device memory (all pointers device pointers, owned by the caller). */
typedef struct {
    int64_t n_rows;          /* N: dense output rows                                    */
    int64_t n_cols;          /* K: dense input columns                                  */
    int32_t R, C;            /* block shape; R | N, C | K                               */
    int64_t nnzb;            /* number of stored blocks                                 */
    const int32_t *indptr;   /* [N/R + 1]                                               */
    const int32_t *indices;  /* [nnzb]                                                  */
    const void *data;        /* [nnzb][R][C] row-major, of type `dtype`                 */
    bsr_dtype dtype;         /* BSR_F32 (float) or BSR_BF16 (uint16 bf16 bit patterns)  */
} bsr_matrix_t;

/*
 * Number of blocks kept at a block density (Sec. 2.1, Eq. 2: the bound tau on the number of
 * nonzero groups): k = floor(density * nb + 0.5) computed in double, clamped to [0, nb].
 * Host only; touches no device.  Errors: BSR_ERR_NULL (k), BSR_ERR_SHAPE (sizes <= 0 or not
 * tiled by R x C), BSR_ERR_ARG (density NaN or outside [0, 1]).
 */
LIBBSR_API bsr_status bsr_prune_count(int64_t N, int64_t K, int32_t R, int32_t C, double density,
                           int64_t *k);

/* Device workspace bytes that bsr_prune_from_dense needs for an N x K weight with R x C blocks
 * (0 if the shape is invalid).  Host only. */
LIBBSR_API size_t bsr_prune_workspace_bytes(int64_t N, int64_t K, int32_t R, int32_t C);

/*
 * Block-magnitude pruning, dense fp32 W -> BSR keeping exactly k blocks (Sec. 2.1, Eq. 2 and
 * Eq. 3, with the l2 norm as the per-block norm; Sec. 2.2 for the BSR layout).
 *   key(i, j) = sum of w^2 over the block, in fp64, summed row r outer, column c inner, from
 *   +0.0 (a NaN key ranks above +inf).  The kept blocks are the first k in the order
 *   (key descending, block id ascending), so the result is unique and equal, bit for bit, to a
 *   CPU computation of the same definition.
 * W: device fp32, N x K with row pitch ldw >= K.
 * k: number of blocks to keep, 0 <= k <= nb (see bsr_prune_count).
 * Outputs (device, caller-allocated): indptr int32[N/R + 1]; indices int32[capacity_blocks];
 *   data float[capacity_blocks * R * C].  The first k entries of indices/data are written; data
 *   holds exact bit copies of W's elements.
 * workspace: device memory of at least bsr_prune_workspace_bytes(N, K, R, C) bytes; its
 *   contents on entry do not matter.  It is in use until the enqueued work completes.
 * Errors: BSR_ERR_NULL, BSR_ERR_SHAPE, BSR_ERR_ARG (k out of range), BSR_ERR_CAPACITY
 *   (capacity_blocks < k), BSR_ERR_WORKSPACE, BSR_ERR_UNSUPPORTED (nb >= 2^31 or
 *   N * ldw >= 2^53), BSR_ERR_ARCH, BSR_ERR_HIP.
 */
LIBBSR_API bsr_status bsr_prune_from_dense(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R,
                                int32_t C, int64_t k, int32_t *indptr, int32_t *indices,
                                float *data, int64_t capacity_blocks, void *workspace,
                                size_t ws_bytes, void *stream);

/* Most blocks (nb = (N / R) * (K / C)) that bsr_prune_from_dense_noalloc handles: its fixed
 * workspace is 12 MiB of device memory per GPU. */
#define BSR_NOALLOC_MAX_BLOCKS (1 << 20)

/*
 * bsr_prune_from_dense without a workspace argument, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Arguments, outputs and result are those of bsr_prune_from_dense (bit-identical to it); the
 * workspace is a fixed array inside the library, one per GPU, held until the process ends, of
 * the size bsr_prune_workspace_bytes() gives for BSR_NOALLOC_MAX_BLOCKS blocks.  The call
 * allocates nothing (no hipMalloc, no library allocation); its first call on a device looks up
 * that device's array with the device current.
 * Every call on one GPU shares that GPU's array, so calls whose work overlaps in time on one
 * GPU (on different streams, or from several threads without ordering) race and must not be
 * issued; calls ordered on one stream are safe.  The array keeps the last call's contents;
 * nothing in it needs to start at zero.
 * Errors: those of bsr_prune_from_dense, with BSR_ERR_WORKSPACE when nb exceeds
 * BSR_NOALLOC_MAX_BLOCKS (checked before anything is enqueued).
 */
LIBBSR_API bsr_status bsr_prune_from_dense_noalloc(const float *W, int64_t N, int64_t K,
                                                   int64_t ldw, int32_t R, int32_t C, int64_t k,
                                                   int32_t *indptr, int32_t *indices,
                                                   float *data, int64_t capacity_blocks,
                                                   void *stream);

/* Pruning variants for the _ex entry points (Sec. 2.1). */
typedef enum {
    BSR_NORM_L2 = 0,  /* block key = sum of w^2 (the l2 group norm, squared)                  */
    BSR_NORM_L1 = 1   /* block key = sum of |w| (the l1 norm, p = 1 in Eq. 1 and Eq. 2)       */
} bsr_norm;
typedef enum {
    BSR_SELECT_GLOBAL = 0,  /* keep the k best blocks of the whole matrix (Eq. 2, tau = k)     */
    BSR_SELECT_PER_ROW = 1  /* keep the k / Nb best blocks of every block-row (Eq. 2 applied to
                               each block-row, tau = k / Nb): every row keeps as many blocks   */
} bsr_select;
typedef struct {
    int32_t norm;    /* a bsr_norm value   */
    int32_t select;  /* a bsr_select value */
} bsr_prune_options_t;

/*
 * bsr_prune_count for a pruning variant: with BSR_SELECT_PER_ROW, k = Nb * k_row where
 * k_row = floor(density * Kb + 0.5) computed in double, clamped to [0, Kb]; otherwise as
 * bsr_prune_count.  opts may be NULL (l2, global).  Host only.  Errors: those of
 * bsr_prune_count, and BSR_ERR_ARG for an unknown norm or selection.
 */
LIBBSR_API bsr_status bsr_prune_count_ex(int64_t N, int64_t K, int32_t R, int32_t C,
                                         double density, const bsr_prune_options_t *opts,
                                         int64_t *k);

/*
 * bsr_prune_from_dense with a choice of block norm and selection (Sec. 2.1):
 *   BSR_NORM_L1: key(i, j) = sum of |w| over the block, in fp64, summed row r outer, column c
 *   inner from +0.0 (|w| is exact in fp64, so the key is bit-identical to a sequential CPU sum;
 *   a NaN key ranks above +inf).  BSR_NORM_L2 is bsr_prune_from_dense's key.
 *   BSR_SELECT_PER_ROW: every block-row keeps its k / Nb blocks that come first in the order
 *   (key descending, block column ascending); k must be a multiple of Nb, and then
 *   indptr[i] = i * (k / Nb).
 * Arguments, outputs, workspace and errors as bsr_prune_from_dense, plus BSR_ERR_ARG for an
 * unknown norm or selection or (per-row) a k that is not a multiple of Nb.  opts may be NULL.
 */
LIBBSR_API bsr_status bsr_prune_from_dense_ex(const float *W, int64_t N, int64_t K, int64_t ldw,
                                              int32_t R, int32_t C, int64_t k,
                                              int32_t *indptr, int32_t *indices, float *data,
                                              int64_t capacity_blocks, void *workspace,
                                              size_t ws_bytes, const bsr_prune_options_t *opts,
                                              void *stream);

/*
 * The BSR product (Sec. 2.2; BERT attention projections, Sec. 2.3):
 *   Y[t][n] = bias[n] + sum over stored blocks p of block-row i = floor(n / R), sum over c < C of
 *             X[t][indices[p] * C + c] * data[p][n - iR][c].
 * Arithmetic is fp32 with fp32 accumulation and fp32 output (bf16 x bf16 products are exact in
 * fp32); the summation order is the kernel's and fixed for a given launch configuration, so
 * repeated calls are bitwise reproducible.  A block-row with no stored blocks gives Y = bias.
 * X: device, T x K (K = W->n_cols) with row pitch ldx, of type x_dtype (BSR_BF16 = uint16 bf16
 *   bit patterns); x_dtype must equal W->dtype.
 * W: host pointer to a bsr_matrix_t describing device arrays.
 * bias: device fp32[N] or NULL.  Y: device fp32, T x N with row pitch ldy.
 * T = 0 is a no-op.  Errors: BSR_ERR_NULL, BSR_ERR_SHAPE, BSR_ERR_ARG (also: the byte range
 *   of Y overlaps X, bias or W's arrays), BSR_ERR_DTYPE, BSR_ERR_UNSUPPORTED, BSR_ERR_ARCH,
 *   BSR_ERR_HIP.
 */
LIBBSR_API bsr_status bsr_spmm(const void *X, bsr_dtype x_dtype, int64_t T, int64_t ldx,
                    const bsr_matrix_t *W, const float *bias, float *Y, int64_t ldy,
                    void *stream);

/* Kernel choice for bsr_spmm_ex (bsr_spmm uses BSR_KERNEL_AUTO: the matrix-core kernel where
 * it has the shape, else the vector-ALU tile kernel, else the generic kernel; the first two
 * stage an input too wide for one LDS tile in column chunks). */
typedef enum {
    BSR_KERNEL_AUTO = 0,     /* the library picks                                           */
    BSR_KERNEL_GENERIC = 1,  /* one thread per output element; every block shape and dtype   */
    BSR_KERNEL_TILED = 2,    /* LDS-staged token tiles on matrix cores; 32x1, 16x1, 32x32,
                                16x16 blocks (BSR_ERR_UNSUPPORTED for other shapes).  An
                                input too wide for one LDS tile (e.g. K = 3072) is staged in
                                column chunks, each row's sum continuing across them         */
    BSR_KERNEL_VALU = 3      /* LDS-staged token tiles on the vector ALUs; 1x1, 1x2, 1x4, 1x8,
                                1x16, 1x32, 2x1, 4x1, 8x1, 2x2, 4x4, 8x8 blocks (fp32; bf16
                                except 1x1; BSR_ERR_UNSUPPORTED for other shapes), column
                                chunks for wide inputs as above                              */
} bsr_kernel;

typedef struct {
    int32_t kernel;     /* a bsr_kernel value                                                */
    int32_t slices;     /* tiled and vector-ALU kernels: block-row slices per 32-token tile;
                           0 = automatic                                                     */
    void *start_event;  /* hipEvent_t or NULL: recorded when the product kernel starts       */
    void *stop_event;   /* hipEvent_t or NULL: recorded when it ends (both or neither)       */
} bsr_spmm_options_t;

/*
 * bsr_spmm with an explicit kernel choice and launch shape (for tests and tuning).  Same
 * arguments, result and errors as bsr_spmm; opts may be NULL (automatic).  Different launch
 * shapes may sum in different orders; each shape is bitwise reproducible.  With an event
 * pair (caller-created hipEvents with timing enabled), the kernel is launched through
 * hipExtLaunchKernel so that hipEventElapsedTime(start, stop) is the kernel's own device time
 * (no event is recorded when T = 0, as nothing is launched).  Extra errors: BSR_ERR_ARG
 * (unknown kernel, slices < 0, only one event given), BSR_ERR_UNSUPPORTED (the forced kernel
 * does not handle this shape, dtype or size).
 */
LIBBSR_API bsr_status bsr_spmm_ex(const void *X, bsr_dtype x_dtype, int64_t T, int64_t ldx,
                                  const bsr_matrix_t *W, const float *bias, float *Y,
                                  int64_t ldy, const bsr_spmm_options_t *opts, void *stream);

/* One product of a batched call: the arguments of one bsr_spmm call. */
typedef struct {
    const void *X;          /* device, T x K, row pitch ldx, of type x_dtype                 */
    bsr_dtype x_dtype;      /* must equal W->dtype                                           */
    int64_t T;              /* tokens (rows of X and Y); 0 = nothing to do for this product  */
    int64_t ldx;            /* row pitch of X in elements, >= K                              */
    const bsr_matrix_t *W;  /* host pointer to the matrix descriptor                         */
    const float *bias;      /* device fp32[N] or NULL                                        */
    float *Y;               /* device fp32, T x N, row pitch ldy                             */
    int64_t ldy;            /* row pitch of Y in elements, >= N                              */
} bsr_spmm_item_t;

/*
 * Several BSR products in as few kernel launches as possible: the projections of one attention
 * layer (Sec. 2.3: Q, K, V and O of BERT), or any set of independent products.  The paper's
 * compiler reuses work across tasks that share a sparse structure (Sec. 2.2, third bullet); here
 * independent products of one block shape share a single launch, up to 8 per launch, which
 * removes the per-launch fixed cost that dominates small token counts.
 * Result: each items[i].Y is what bsr_spmm_ex(items[i], opts) computes with the same kernel and
 * slice count.  With opts->slices = 0 the automatic slice count considers the token tiles of
 * every product in the launch, so it can differ from a single call's choice (the results then
 * differ only in fp32 summation order).  Products are independent and may run in any order or
 * concurrently: no Y may overlap another product's X, W arrays, bias or Y.  With an event pair
 * in opts, the start event is recorded at the start of the first kernel and the stop event at
 * the end of the last one.  n_items = 0 (or all T = 0) is a no-op.
 * Errors: as bsr_spmm_ex for the first invalid item (nothing is launched if any item is
 *   invalid); BSR_ERR_ARG for n_items < 0, and for a Y that overlaps another product's X,
 *   bias, W arrays or Y (checked on the host, before anything is launched); BSR_ERR_NULL for
 *   items = NULL with n_items > 0.
 */
LIBBSR_API bsr_status bsr_spmm_batched(const bsr_spmm_item_t *items, int32_t n_items,
                                       const bsr_spmm_options_t *opts, void *stream);

/*
 * The arithmetic of a planned product (fixed when the plan is prepared).
 *   BSR_ARITH_AUTO:   BSR_ARITH_NATIVE.
 *   BSR_ARITH_NATIVE: products in the data's own type on the matrix cores (fp32 data on fp32
 *                     MFMA, bf16 data on bf16 MFMA), fp32 accumulate; Y is bit-identical to
 *                     the same product without a plan.
 *   BSR_ARITH_BF16X3: fp32 data only (32x1 blocks): every fp32 operand x is the sum of three
 *                     bf16 pieces x0 + x1 + x2 (x0 = x with its low 16 bits cleared, x1 the
 *                     same of the remainder, x2 what is left; |x1| < 2^-7 |x|,
 *                     |x2| < 2^-14 |x|), exact for |x| >= 2^-103 (below that the last piece
 *                     drops bits under 2^-126).  Each product x w is formed from the six
 *                     cross terms xi wj with i + j <= 2, each exact in fp32, on bf16 MFMA
 *                     with fp32 accumulate; the three terms left out are below 2^-20 |x w|.
 *                     Y therefore meets the same accuracy bound as fp32 arithmetic
 *                     (|err| <= 1e-5 sum |x||w| + 1e-6 in the tests), in a different
 *                     summation order (not bit-identical to NATIVE).  Integer-valued inputs
 *                     with |x|, |w| < 256 are their own first pieces, so integer results stay
 *                     exact.  Non-finite inputs: an infinite x or w gives NaN where fp32
 *                     arithmetic gives an infinity.
 */
typedef enum { BSR_ARITH_AUTO = 0, BSR_ARITH_NATIVE = 1, BSR_ARITH_BF16X3 = 2 } bsr_arith;

/*
 * A per-matrix product plan: the work of a BSR product that depends only on the matrix,
 * prepared once and reused by every product with that matrix (the paper's compiler keeps a
 * buffer of sparse operators and reuses tasks whose sparse structure is identical, Sec. 2.2,
 * third bullet).  The plan cuts every block-row into units of unit_blocks consecutive stored
 * blocks (the last unit of a row padded with zero blocks) and stores
 *   - uptr int32[N/R + 1]: the first unit of every block-row (a row pointer over units);
 *   - the units' block columns and weights, packed in the order the matrix cores consume them,
 *     so one 16-byte load per lane fetches a unit's operands;
 * in caller-owned device memory.  A plan of BSR_ARITH_NATIVE arithmetic computes the same sums
 * in the same order as the product without one (bit-identical Y); it only reads its operands
 * faster.  A plan of BSR_ARITH_BF16X3 stores every weight as its three bf16 pieces and forms
 * the products as described at bsr_arith.  Plans exist for 32x1 blocks (fp32 and bf16 data);
 * bsr_plan_bytes reports BSR_ERR_UNSUPPORTED for other shapes.
 * The struct is filled by bsr_plan_prepare and read by the planned products; it records the
 * matrix it was prepared for, and a product whose matrix differs (shape, block shape, dtype,
 * nnzb or array addresses) is rejected with BSR_ERR_ARG.  The plan's memory must stay
 * allocated and unchanged while products use it; after the matrix's arrays change (same
 * addresses, new contents), prepare the plan again.  The library checks the struct against
 * the matrix, not the contents of mem: the products trust what bsr_plan_prepare wrote there
 * (every column the plan stores is clamped into the X tile when it is packed, so a plan
 * whose matrix indices were out of range still reads only inside the tile).
 */
typedef struct {
    void *mem;                /* device memory holding the plan (caller-owned)                */
    size_t bytes;             /* its size, >= bsr_plan_bytes()                                 */
    int64_t n_rows, n_cols, nnzb;                    /* the matrix it was prepared for        */
    int32_t R, C;
    int32_t dtype;
    const int32_t *indptr;
    const int32_t *indices;
    const void *data;
    int32_t unit_blocks;      /* stored blocks per unit                                        */
    int64_t max_units;        /* units the layout reserves: ceil(nnzb / unit_blocks) + N / R   */
    int64_t uptr_offset;      /* byte offsets into mem of the three arrays                     */
    int64_t col_offset;
    int64_t val_offset;
    int32_t arith;            /* the plan's arithmetic, resolved: BSR_ARITH_NATIVE or _BF16X3  */
} bsr_plan_t;

/* Device bytes a plan for W needs (host only).  Errors: BSR_ERR_NULL, those of a malformed
 * descriptor (BSR_ERR_SHAPE, BSR_ERR_ARG), BSR_ERR_UNSUPPORTED (no planned kernel for the
 * block shape, or sizes past int32 offsets). */
LIBBSR_API bsr_status bsr_plan_bytes(const bsr_matrix_t *W, size_t *bytes);

/* bsr_plan_bytes for a plan of the given arithmetic (a bsr_arith value; bsr_plan_bytes is
 * BSR_ARITH_AUTO).  Extra errors: BSR_ERR_ARG (unknown arithmetic), BSR_ERR_UNSUPPORTED
 * (BSR_ARITH_BF16X3 with bf16 data, or with more than 16383 block columns). */
LIBBSR_API bsr_status bsr_plan_bytes_ex(const bsr_matrix_t *W, int32_t arith, size_t *bytes);

/*
 * Prepare the plan of W in `mem` (device, caller-owned, at least bsr_plan_bytes(W) bytes, not
 * overlapping W's arrays) and fill *plan.  Two kernels on `stream`: a scan of the per-row unit
 * counts, then the packing of every unit's columns and weights.  Errors: those of
 * bsr_plan_bytes, BSR_ERR_NULL (mem, plan), BSR_ERR_WORKSPACE (bytes too small), BSR_ERR_ARG
 * (mem overlapping W's arrays), BSR_ERR_ARCH, BSR_ERR_HIP.
 */
LIBBSR_API bsr_status bsr_plan_prepare(const bsr_matrix_t *W, void *mem, size_t bytes,
                                       bsr_plan_t *plan, void *stream);

/* bsr_plan_prepare with the plan's arithmetic (a bsr_arith value; bsr_plan_prepare is
 * BSR_ARITH_AUTO), recorded in plan->arith.  Errors: those of bsr_plan_bytes_ex and of
 * bsr_plan_prepare. */
LIBBSR_API bsr_status bsr_plan_prepare_ex(const bsr_matrix_t *W, int32_t arith, void *mem,
                                          size_t bytes, bsr_plan_t *plan, void *stream);

/*
 * bsr_spmm_batched with a plan per product (plans may be NULL, or plans[i] NULL for a product
 * without one).  A planned product runs on the planned form of the matrix-core kernel in its
 * plan's arithmetic: with BSR_ARITH_NATIVE it gives the same Y, bit for bit, as the same call
 * without plans, with one exception: when a launch has more token tiles than the GPU has CUs
 * and holds an even number of planned products in which items 2i and 2i + 1 read the same X
 * (same pointer, T, ldx and column count), those two run paired, one workgroup serving a token
 * tile of both, and sum their rows in another order (same accuracy; integer-valued results
 * stay exact).  A paired product's Y is still bitwise reproducible for the same call.  Products
 * with and without plans, or with plans of different arithmetic, never share a launch.
 * Errors: those of bsr_spmm_batched, and BSR_ERR_ARG for a plan that does not describe its
 * product's matrix or whose memory overlaps a Y.
 */
LIBBSR_API bsr_status bsr_spmm_batched_planned(const bsr_spmm_item_t *items,
                                               const bsr_plan_t *const *plans, int32_t n_items,
                                               const bsr_spmm_options_t *opts, void *stream);

/*
 * Scaled dot-product attention of the BERT attention block (Sec. 2.3 prunes BERT's attention
 * weights; its Q, K, V and output projections are the BSR products above):
 *   O[b*seq + s][h*64 + d] = sum_j p_j V[b*seq + j][h*64 + d],
 *   p_j = softmax over j < seq of scale * sum_e Q[b*seq + s][h*64 + e] * K[b*seq + j][h*64 + e].
 * Rows are tokens (batch-major), head h owns columns h*64 .. h*64 + 63; no mask.  fp32 inputs,
 * fp32 arithmetic (online softmax with expf), fp32 output.
 * Q, K, V: device fp32 with row pitches ldq, ldk, ldv >= heads * 64, 16-byte aligned bases and
 *   pitches that are multiples of 4.  O: device fp32, row pitch ldo >= heads * 64; it must not
 *   overlap Q, K or V.  head_dim must be 64.  batch = 0 or seq = 0 is a no-op.
 * Errors: BSR_ERR_NULL, BSR_ERR_SHAPE (negative sizes, heads < 1, a pitch below heads * 64),
 *   BSR_ERR_ARG (scale not finite), BSR_ERR_UNSUPPORTED (head_dim != 64, misaligned inputs,
 *   batch or heads above 65535), BSR_ERR_ARCH, BSR_ERR_HIP.
 */
LIBBSR_API bsr_status bsr_attention(const float *Q, int64_t ldq, const float *K, int64_t ldk,
                                    const float *V, int64_t ldv, float *O, int64_t ldo,
                                    int32_t batch, int32_t seq, int32_t heads, int32_t head_dim,
                                    float scale, void *stream);

/*
 * The same matrix stored with finer R2 x C2 blocks, R2 a divisor of W->R and C2 of W->C (the
 * Sec. 2.2 layout at a smaller block size, as SciPy converts a BSR matrix to one).  With
 * a = R / R2 and b = C / C2, the q-th of the n stored blocks of block-row i (column
 * j = indices[p]) is cut into a x b pieces; piece (r, s) holds rows r*R2 .. r*R2 + R2 - 1 and
 * columns s*C2 .. s*C2 + C2 - 1 of the block and is stored
 *   in fine block-row i*a + r, at position indptr[i]*a*b + r*n*b + q*b + s, column j*b + s,
 * so indptr_out[i*a + r] = indptr[i]*a*b + r*n*b and every fine block-row keeps its columns
 * ascending.  Values are copied bit for bit; a piece that is all zeros stays stored.  A matrix
 * pruned with a large block (64 x 64, 1 x 64 ... 1 x 384, 64 x 1) then runs on the product
 * kernels of a divisor shape (32 x 32, 1 x 32, 32 x 1) with unchanged results up to the order
 * of the sums.
 * Outputs (device, caller-owned, not overlapping W's arrays or each other): indptr_out
 *   int32[N/R2 + 1],
 * indices_out int32[nnzb*a*b], data_out [nnzb*a*b][R2][C2] elements of W's dtype.  The fine
 * matrix is {N, K, R2, C2, nnzb*a*b, indptr_out, indices_out, data_out, W->dtype}.
 * Errors: BSR_ERR_NULL, BSR_ERR_ARG (W's dtype or nnzb, or overlapping byte ranges of the
 *   arrays), BSR_ERR_SHAPE (W's shape, or R2 or C2
 *   not a positive divisor of R or C), BSR_ERR_UNSUPPORTED (more than 2^31 - 1 fine blocks),
 *   BSR_ERR_ARCH, BSR_ERR_HIP.
 */
LIBBSR_API bsr_status bsr_reblock(const bsr_matrix_t *W, int32_t R2, int32_t C2,
                                  int32_t *indptr_out, int32_t *indices_out, void *data_out,
                                  void *stream);

/*
 * Expand an fp32 BSR matrix to dense (Sec. 2.2 layout): out[n][k] = the stored element covering
 * (n, k), or +0.0 where no block is stored.  out: device fp32, N x K with row pitch ldo >= K.
 * Errors: BSR_ERR_NULL, BSR_ERR_SHAPE, BSR_ERR_DTYPE (bf16 data), BSR_ERR_UNSUPPORTED,
 *   BSR_ERR_ARCH, BSR_ERR_HIP.
 */
LIBBSR_API bsr_status bsr_to_dense(const bsr_matrix_t *W, float *out, int64_t ldo, void *stream);

/*
 * fp32 -> bf16, round to nearest with ties to even; NaN stays a quiet NaN (its upper 16 bits
 * with the quiet bit set); overflow rounds to infinity.  Used to feed the bf16 product with
 * bf16 activations and BSR data.  src, dst: device arrays of n elements (dst as uint16).
 * Errors: BSR_ERR_NULL, BSR_ERR_SHAPE (n < 0), BSR_ERR_ARCH, BSR_ERR_HIP.
 */
LIBBSR_API bsr_status bsr_cast_f32_bf16(const float *src, uint16_t *dst, int64_t n, void *stream);

/*
 * One gradient step of the iterative projection for Eq. 2 (Sec. 2.1: minimise a loss under a
 * bound on the number of nonzero blocks).  With the layer-output reconstruction loss on
 * calibration activations X (T x K), f(W) = 1/2 tr((W - W0) H (W - W0)^T) with
 * H = X^T X / T, projected gradient descent (iterative hard thresholding) takes
 *   W <- P_k(W - eta (W - W0) H),
 * where P_k is the block prune (bsr_prune_from_dense with k blocks).  The two products of the
 * gradient are bsr_spmm calls with the symmetric H as their X operand: G = H W^T (W the
 * current BSR iterate) and C0 = H W0^T (W0 stored with all its blocks).  This call forms
 *   V[n][j] = W[n][j] - eta * (G[j][n] - C0[j][n]),   n < N, j < K,
 * rounding the subtraction, the product and the final subtraction to fp32 one at a time (no
 * fused multiply-add).  W: device fp32 N x K (the iterate, dense, row pitch ldw >= K); G, C0:
 * device fp32 K x N (row pitches ldg, ldc >= N); V: device fp32 N x K (ldv >= K), which may be
 * W itself (then ldv == ldw) but must not overlap G or C0.  Errors: BSR_ERR_SHAPE (N or K < 0,
 * a pitch too small), BSR_ERR_ARG (non-finite eta; V overlapping an input other than as W
 * itself), BSR_ERR_NULL, BSR_ERR_UNSUPPORTED (N >= 2^37, K > 4194240, offsets past 2^53),
 * BSR_ERR_ARCH, BSR_ERR_HIP.
 */
LIBBSR_API bsr_status bsr_iht_update(const float *W, int64_t ldw, const float *G, int64_t ldg,
                                     const float *C0, int64_t ldc, float eta, int64_t N,
                                     int64_t K, float *V, int64_t ldv, void *stream);

/* Static, human-readable name of a status code. */
LIBBSR_API const char *bsr_status_str(bsr_status s);

/* Text of the last HIP error seen by this thread's libbsr calls ("" if none). */
LIBBSR_API const char *bsr_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LIBBSR_H */
