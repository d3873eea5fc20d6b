/*
 * gnnspmm.h -- C ABI of the MI355X (gfx950) GNN-aggregation SpMM library.
 *
 * The library computes Y = A.X, the neighbourhood aggregation of a GNN layer
 * (arXiv 2111.00352, Sec. 2.1: A is the sparse N x N adjacency, X the dense
 * N x d node-feature matrix), with A held in one of the sparse storage
 * formats of Sec. 2.2 (COO, CSR, CSC, DIA, BSR) or in padded row-packed ELL.
 * Around the kernels it provides what the paper's runtime does before each
 * GNN layer (Sec. 4, Sec. 4.6): extraction of the matrix features of Table 2
 * (Sec. 4.4), min-max normalisation and a tree-ensemble format predictor
 * (Sec. 4.1, 4.4), conversion to the chosen format when it differs from the
 * one already held (Sec. 4), and dispatch of that format's kernel.
 *
 * Conventions for every call:
 *   - Pointers marked [dev] are device pointers (hipMalloc'd or torch CUDA
 *     tensors); [host] pointers are ordinary host memory.
 *   - Index arrays are int32, values fp32.  Matrices must satisfy
 *     n_rows, n_cols < 2^31 and nnz < 2^31.
 *   - Dense matrices are row-major with a leading dimension (elements
 *     between consecutive rows) ld >= F.
 *   - gs_stream is a hipStream_t (NULL = the legacy null stream).  Work is
 *     enqueued on it; calls that need device results on the host say so.
 *   - Every int-returning call returns GS_OK (0) or a negative gs_status.
 *     On error every output handle is set to NULL, nothing is leaked, and
 *     gs_last_error() describes the failure.  No C++ exception crosses the
 *     ABI.
 *   - The library never writes to caller-owned inputs.
 */
#ifndef GNNSPMM_H
#define GNNSPMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void *gs_stream; /* hipStream_t */

/* Storage formats (Sec. 2.2; ELL = rows packed to the longest row). */
typedef enum {
    GS_COO = 0,
    GS_CSR = 1,
    GS_ELL = 2,
    GS_DIA = 3,
    GS_BSR = 4,
    GS_CSC = 5,
    GS_NUM_FORMATS = 6
} gs_format;

typedef enum {
    GS_OK = 0,
    GS_ERR_INVALID_ARG = -1,   /* null pointer, bad enum, F <= 0, ld < F, sizes out of range */
    GS_ERR_INDEX = -2,         /* a row/col index outside [0,n_rows) x [0,n_cols) */
    GS_ERR_DUPLICATE = -3,     /* two entries with the same (row, col) */
    GS_ERR_EXPLICIT_ZERO = -4, /* a stored value equal to +0.0f or -0.0f */
    GS_ERR_INFEASIBLE = -5,    /* padded storage would exceed max_bytes */
    GS_ERR_OOM = -6,           /* the allocator returned NULL */
    GS_ERR_HIP = -7,           /* a HIP runtime call failed */
    GS_ERR_MODEL = -8,         /* predictor model missing or malformed */
    GS_ERR_UNSUPPORTED = -9    /* a valid request the library does not handle */
} gs_status;

/* A sparse matrix in coordinate form, as PyTorch-Geometric hands it over
 * (Sec. 2.2, COO).  All three arrays are [dev], nnz entries each, borrowed
 * for the duration of the call (until the enqueued work has completed).
 * Order is arbitrary unless assume_canonical is set in gs_build_opts.
 * Errors are reported with precedence INDEX > EXPLICIT_ZERO > DUPLICATE. */
typedef struct {
    int64_t n_rows, n_cols, nnz;
    const int32_t *row; /* [dev] */
    const int32_t *col; /* [dev] */
    const float *val;   /* [dev] */
} gs_coo;

typedef struct {
    int32_t bsr_block;        /* BSR block edge b, 1..64; 0 -> 16 */
    int32_t assume_canonical; /* 1: caller guarantees (row,col)-sorted, no duplicates
                                 (still validated; an unsorted input is then an error) */
    uint64_t max_bytes;       /* cap on a padded format's device bytes; 0 -> 8 GiB */
} gs_build_opts;

/* Optional device allocator (e.g. PyTorch's caching allocator).  alloc must
 * return memory usable on the given stream, aligned to 256 bytes, or NULL.  The hooks must be
 * stream-ordered: free(p, s) can be called while work already enqueued on s
 * still uses p, so p may go to later work on s, but to other streams only
 * once that work has completed (PyTorch's caching allocator and
 * hipFreeAsync behave so).  NULL hooks (the default) mean hipMalloc and a
 * synchronisation of s before hipFree. */
typedef struct {
    void *(*alloc)(size_t bytes, gs_stream s, void *ctx);
    void (*free)(void *p, gs_stream s, void *ctx);
    void *ctx;
} gs_allocator;

typedef struct gs_matrix_ *gs_matrix; /* opaque; owns its device arrays (the format's arrays are
                                         immutable once built) and one SpMM workspace */
typedef struct gs_ctx_ *gs_ctx;       /* opaque; per-adjacency feature/format cache + selector */

/* Installs the device allocator for all later allocations (NULL restores
 * hipMalloc/hipFree).  Memory always goes back through the hooks that
 * allocated it, so handles built before a change stay valid; hooks (and
 * their ctx) must therefore remain callable until every handle and
 * context that allocated through them has been destroyed.  Not
 * thread-safe against concurrent library calls. */
int gs_set_allocator(const gs_allocator *a);

/* Builds A in format fmt on the device (Sec. 2.2; conversion, Sec. 4).
 * Validates, canonicalises (sorts by (row, col) when needed), builds CSR and
 * from it the requested layout, each in the canonical form:
 *   COO  row[nnz], col[nnz], val[nnz] sorted by (row, col)
 *   CSR  row_ptr[n_rows+1], col[nnz], val[nnz]
 *   CSC  col_ptr[n_cols+1], row[nnz], val[nnz] sorted by (col, row): the
 *        CSR of the transpose
 *   ELL  K = longest row; ell_col[K*n_rows], ell_val[K*n_rows], slot (i,k) at
 *        k*n_rows+i; padding col = -1, val = +0.0f
 *   DIA  offsets[N_diags] ascending distinct (col-row); data[N_diags*n_rows],
 *        data[d*n_rows+i] = A[i, i+offsets[d]] or +0.0f
 *   BSR  b = bsr_block; block_ptr[ceil(n_rows/b)+1]; block_col[nb] ascending per
 *        block row; block_val[nb*b*b], A[r,c] at blk*b*b + (r%b)*b + c%b,
 *        every other slot +0.0f (the matrix is zero-padded to whole blocks)
 * opts may be NULL (defaults).  Synchronises s once (sizes are needed on the
 * host).  On GS_ERR_INFEASIBLE *bytes_required (if non-NULL) holds the bytes
 * the format would need; on success it holds the bytes allocated. */
int gs_build_format(const gs_coo *A, int fmt, const gs_build_opts *opts, gs_stream s,
                    gs_matrix *out, uint64_t *bytes_required);

/* Converts an already built matrix into another format without re-checking
 * it.  Same layouts, options and errors as gs_build_format. */
int gs_convert(gs_matrix A, int fmt, const gs_build_opts *opts, gs_stream s, gs_matrix *out,
               uint64_t *bytes_required);

/* SpMM, Sec. 2.1: Y = A.X, Y overwritten (Y[i,:] = 0 for an empty row i).
 * X [dev] n_cols x F, row-major, leading dimension ldx >= F; Y [dev]
 * n_rows x F, leading dimension ldy >= F; columns F..ld-1 are not touched.
 * F is at most 2^24 (GS_ERR_UNSUPPORTED beyond), and each operand's span
 * ((rows - 1) * ld + F floats) must be addressable (GS_ERR_INVALID_ARG
 * otherwise).  X and Y must not overlap.  fp32 in and out; products and sums in fp32
 * (fused multiply-add), with every sequential chain kept short enough that
 * |Y - A.X| <= 1e-5 (|A|.|X|) + 1e-6 elementwise.  Deterministic: the same
 * inputs give bit-identical Y.  CSC is the exception: its columns scatter
 * into the rows of Y, so the products (exact in fp64) are added with fp64
 * atomics in a workspace and rounded to fp32 once; the order of the fp64
 * additions varies, which can change an fp32 result only where an fp64
 * sum sits on an fp32 rounding boundary.  Fully asynchronous on s; the
 * first call with a larger F than before may allocate a workspace (in
 * stream order).  That workspace (partial sums of split rows, COO carries,
 * the CSC accumulator) belongs to the handle: SpMM calls on one handle must
 * not overlap in time (issue them on one stream or order them); different
 * handles are independent. */
int gs_spmm(gs_matrix A, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
            gs_stream s);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): gs_spmm
 * with the same arguments and the same result, bit for bit, that never calls
 * the allocator.  The F-dependent workspace that gs_spmm keeps in the handle
 * (partial sums of split CSR rows, the CSC fp64 accumulator) comes instead
 * from a fixed array of GS_NOALLOC_SCRATCH_BYTES in device memory, one per
 * device, reserved when the library's code is loaded on that device and held
 * until the process ends.  Every call on one device shares that device's
 * array and leaves it in an undefined state: calls that may overlap in time
 * on one device (other streams, other threads) race, so order them.
 * Supported for CSR, ELL, DIA, BSR and CSC handles built by gs_build_format
 * or gs_convert.  Errors: GS_ERR_UNSUPPORTED for a COO handle (its range
 * tables are built, and allocated, per launch shape on first use) and when
 * the workspace would exceed GS_NOALLOC_SCRATCH_BYTES (CSR: at most 4 * F
 * bytes per 128 entries of the rows longer than 128 entries, as many as the
 * row plan cuts into chunks; CSC: 8 * n_rows * F bytes); otherwise as
 * gs_spmm.  Asynchronous on s. */
#define GS_NOALLOC_SCRATCH_BYTES (64u << 20)
int gs_spmm_noalloc(gs_matrix A, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                    gs_stream s);

/* Writes the canonical COO of A (sorted by (row, col)) into caller-allocated
 * [dev] arrays of nnz entries each.  For padded formats, padding slots are
 * dropped (ELL col == -1; DIA/BSR value == 0 or outside the matrix).
 * Asynchronous on s. */
int gs_to_coo(gs_matrix A, int32_t *row, int32_t *col, float *val, gs_stream s);

typedef struct {
    int32_t format;        /* gs_format */
    int32_t bsr_block;     /* b for BSR, else 0 */
    int64_t n_rows, n_cols, nnz;
    int64_t param;         /* ELL: K, DIA: N_diags, BSR: number of blocks, else 0 */
    uint64_t device_bytes; /* bytes of the format's arrays (excluding workspaces) */
} gs_matrix_info;

int gs_get_info(gs_matrix A, gs_matrix_info *info);

/* Raw arrays of a built matrix, for inspection and bit-exact comparison.
 * which: 0 = row_ptr|row|ell_col|offsets|block_ptr|col_ptr,
 *        1 = col|ell_val|data|block_col|row (CSC), 2 = val|block_val
 *        (see gs_build_format for per-format meaning).
 * *dev_ptr receives a [dev] pointer owned by A, *bytes its size. */
int gs_get_array(gs_matrix A, int which, const void **dev_ptr, uint64_t *bytes);

/* Copies raw array `which` (as in gs_get_array) into caller memory dst [dev]
 * of dst_bytes >= the array's size.  Asynchronous on s. */
int gs_copy_array(gs_matrix A, int which, void *dst, uint64_t dst_bytes, gs_stream s);

/* Frees A's device arrays and workspace through the hooks that allocated
 * them, in the order of the stream A was built on.  When A was last read on
 * another stream (gs_spmm, gs_spmm_noalloc, gs_to_coo, gs_copy_array), the
 * call first waits for that work to finish, so no later allocation on the
 * build stream can reuse the memory under it.  Work captured into a graph
 * is not tracked: destroy A only after the graph's last replay.  NULL is
 * ignored. */
void gs_destroy(gs_matrix A);

/* Matrix features of Table 2 (Sec. 4.4), extracted on the device from the
 * canonical form of A.  Integer aggregates are exact; the doubles are
 * computed on the host from them in a fixed operation order:
 *   dev = sqrt((n*S2 - Z^2) / (n*n)) with the numerator formed exactly,
 *   ER_DIA = Z/(N_diags*R), ER_CD = Z/(C*max_CD), bounce = sum|count
 *   difference of adjacent rows (columns)| / (R-1) (C-1), density = Z/(R*C),
 *   cv = dev_RD/aver_RD, max_mu = max_RD - aver_RD; ratios with a zero
 *   denominator are 0.  f[] is F1..F19 in Table 2 order.  n_blocks16 is
 *   the number of distinct (row/16, col/16) pairs (a BSR footprint input for
 *   the selector, not in Table 2).  Synchronises s. */
typedef struct {
    int64_t n_rows, n_cols, nnz, n_diags, max_rd, min_rd, max_cd, min_cd;
    uint64_t sum_rd2, sum_cd2, bounce_r, bounce_c;
    int64_t n_blocks16;
    double f[19];
} gs_features;

int gs_extract_features(const gs_coo *A, const gs_build_opts *opts, gs_stream s,
                        gs_features *out);

/* Same, from an already built matrix (any format). */
int gs_matrix_features(gs_matrix A, gs_stream s, gs_features *out);

/* ---- per-layer selection and dispatch (Sec. 4, Sec. 4.6) ---- */

typedef enum {
    GS_SEL_MODEL = 0,   /* tree-ensemble predictor over the normalised features */
    GS_SEL_PROFILE = 1, /* run every feasible format once and keep the fastest */
    GS_SEL_FIXED = 2    /* always the format in `fixed` */
} gs_sel_mode;

typedef struct {
    int32_t mode;           /* gs_sel_mode */
    int32_t fixed;          /* gs_format for GS_SEL_FIXED */
    const char *model_path; /* [host] model file, read only for GS_SEL_MODEL; NULL = built-in model */
    uint64_t max_bytes;     /* formats whose padded size exceeds this are never chosen; 0 -> 8 GiB */
    int32_t bsr_block;      /* 0 -> 16 */
    int32_t profile_reps;   /* timed runs per format for GS_SEL_PROFILE; 0 -> 3 */
    uint32_t formats;       /* candidates of MODEL and PROFILE: bit f set = gs_format f;
                               0 -> every format (the paper's whole pool) */
    double mem_weight;      /* 1 - w of Eq. 1 (Sec. 4.3): the weight of the memory footprint against
                               the running time, in [0, 1]; 0 -> time only (w = 1).  PROFILE picks
                               the candidate with the smallest w R + (1 - w) M, R its measured time
                               and M its device bytes, each min-max scaled over this (matrix, F)'s
                               feasible candidates; O within 1e-4 of the smallest counts as tied
                               (Fig. 6 caption) and the first in the order CSR, COO, ELL, DIA, BSR,
                               CSC is taken.  MODEL needs a model trained for the same w (its "w" line, 1
                               when absent): otherwise gs_ctx_create fails with GS_ERR_MODEL.  FIXED
                               ignores it.  Outside [0, 1] or NaN: GS_ERR_INVALID_ARG. */
} gs_selector_opts;

int gs_ctx_create(const gs_selector_opts *o, gs_ctx *out);
void gs_ctx_destroy(gs_ctx c); /* frees every cached matrix */

/* One GNN layer's aggregation with format selection: Y = A.X with A in the
 * format the selector picks for (A, F).  `key` names the adjacency: the
 * first call with a key extracts features and builds the canonical form
 * (synchronising s); later calls with the same key reuse them and assume A
 * is unchanged.  The format is decided once per (key, F) (the predictor
 * sees F as an input) and reused by later calls, and a format is converted
 * at most once per key, as the paper converts only when the chosen format
 * differs from the previous layer's or epoch's.  *chosen (may be NULL) receives the format used.
 * Arguments otherwise as gs_spmm.  A gs_ctx is not thread-safe. */
int gs_select_and_run(gs_ctx c, uint64_t key, const gs_coo *A, const float *X, int64_t ldx,
                      float *Y, int64_t ldy, int64_t F, gs_stream s, int32_t *chosen);

/* What the selector would choose for (key, F) without running the SpMM.
 * Same caching as gs_select_and_run (the first call for a key synchronises). */
int gs_select(gs_ctx c, uint64_t key, const gs_coo *A, int64_t F, gs_stream s, int32_t *chosen);

/* Host-side statistics of the last selection made through c: time spent in
 * feature extraction, prediction and conversion (seconds, wall clock;
 * features and conversion as measured on the first call for the key /
 * format, prediction as spent in this call, a cache lookup after the first
 * call for a (key, F)). */
typedef struct {
    double t_features, t_predict, t_convert;
    int32_t chosen;
    int32_t feasible_mask;  /* bit f set if format f fits max_bytes */
    double scores[GS_NUM_FORMATS]; /* per-format predictor scores (MODEL) or seconds (PROFILE) */
} gs_select_stats;

int gs_ctx_stats(gs_ctx c, gs_select_stats *out);

/* Thread-local description of the last error (never NULL). */
const char *gs_last_error(void);

/* ABI version of this header (incremented on incompatible change). */
int gs_abi_version(void);
#define GS_ABI_VERSION 3

#ifdef __cplusplus
}
#endif
#endif /* GNNSPMM_H */
