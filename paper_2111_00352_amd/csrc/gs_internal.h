// Internal declarations of the gfx950 SpMM library: matrix handle layout,
// allocation, error reporting and the kernel launchers shared between files.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/gnnspmm.h"

namespace gs {

// ----------------------------------------------------------------- errors

void set_error(const char *fmt, ...) __attribute__((format(printf, 1, 2)));

struct Error {
    int code;
};

// Throws Error{GS_ERR_HIP} with the HIP message when e != hipSuccess.
void hip_check(hipError_t e, const char *what);
#define GS_HIP(call) ::gs::hip_check((call), #call)

[[noreturn]] void fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

// Runs f, converting Error / std::bad_alloc into status codes.
template <class Fn>
int guarded(Fn &&f)
{
    try {
        f();
        return GS_OK;
    } catch (const Error &e) {
        return e.code;
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed");
        return GS_ERR_OOM;
    } catch (...) {
        set_error("unexpected internal exception");
        return GS_ERR_INVALID_ARG;
    }
}

// --------------------------------------------------------------- memory

// Allocates through the hooks installed now (recorded in *used) and frees
// through the hooks recorded at allocation, whatever is installed later.
void *dev_alloc(size_t bytes, hipStream_t s, gs_allocator *used);  // throws Error{GS_ERR_OOM}
void dev_free(void *p, hipStream_t s, const gs_allocator &used);

// A device buffer freed when the owner goes away.
struct DevBuf {
    void *p = nullptr;
    size_t bytes = 0;
    hipStream_t s = nullptr;
    gs_allocator how{};  // the hooks that allocated p
    DevBuf() = default;
    DevBuf(const DevBuf &) = delete;
    DevBuf &operator=(const DevBuf &) = delete;
    DevBuf(DevBuf &&o) noexcept : p(o.p), bytes(o.bytes), s(o.s), how(o.how) { o.p = nullptr; o.bytes = 0; }
    DevBuf &operator=(DevBuf &&o) noexcept
    {
        if (this != &o) {
            reset();
            p = o.p; bytes = o.bytes; s = o.s; how = o.how;
            o.p = nullptr; o.bytes = 0;
        }
        return *this;
    }
    ~DevBuf() { reset(); }
    void alloc(size_t n, hipStream_t st)
    {
        reset();
        s = st;
        p = n ? dev_alloc(n, st, &how) : nullptr;
        bytes = n;
    }
    void reset()
    {
        if (p) dev_free(p, s, how);
        p = nullptr;
        bytes = 0;
    }
    template <class T> T *as() const { return static_cast<T *>(p); }
};

struct WorkArea;

// ------------------------------------------------------------ matrix handle

}  // namespace gs

struct gs_matrix_ {
    int fmt = GS_CSR;
    int64_t R = 0, C = 0, Z = 0;
    hipStream_t stream = nullptr;  // stream the arrays were allocated on

    // COO (row, col, val) and CSR (row_ptr, col, val) share col/val; CSC
    // keeps its col_ptr / row indices / values in row_ptr / col / val (it is
    // the CSR of the transpose).
    gs::DevBuf row, row_ptr, col, val;
    // ELL
    int64_t K = 0;
    gs::DevBuf ell_col, ell_val;
    // DIA
    int64_t ND = 0;
    gs::DevBuf offsets, dia;
    // BSR
    int32_t b = 0;
    int64_t nb = 0;
    gs::DevBuf bptr, bcol, bval, bmask;  // bmask: per block 64-bit mask of nonzero columns
    int64_t n_dense_blocks = 0;
    // BSR(16) hybrid plan: the dense blocks of each block row (indices into
    // the block arrays; hyb_dptr[nbr+1]) and the entries of every other block
    // as a CSR of their own (hyb_rrp[R+1], hyb_rcol, hyb_rval)
    bool hyb_planned = false;
    int64_t hyb_ndense = 0, hyb_nrest = 0;
    gs::DevBuf hyb_dptr, hyb_didx, hyb_rrp, hyb_rcol, hyb_rval;

    // Kernel plans built once per matrix.
    // CSR: rows longer than the short-row limit, split into chunks.
    int csr_long_thr = 0, csr_chunk = 0;
    int64_t n_long_rows = 0, n_long_chunks = 0;
    gs::DevBuf long_rows;    // int32 row ids, n_long_rows
    gs::DevBuf long_first;   // int32 [n_long_rows+1] -> first partial slot of each long row
    gs::DevBuf csr_items;    // int4 {row, start, len, slot} work items
    int64_t n_items = 0;
    int64_t n_short = 0;     // short items (after the n_long_chunks chunk items)
    int64_t n_medium_rows = 0, n_medium_chunks = 0;  // long rows of at most csr_wg_thr entries
    int csr_wg_thr = 0;
    bool csr_sorted = false; // items ordered by decreasing length
    bool csr_grouped = false; // group tier: short items may be rows of up to kCsrGroupRow entries
    bool csr_planned = false; // plan_csr has run (a CSR built only for its features has no plan)
    // CSR: column indices tagged with their column's reference class (bit
    // length of its entry count) in bits 27..30 (made by the first SpMM that
    // gathers by class), each column's class, and the number of columns in
    // each class; empty when the matrix does not use classes
    gs::DevBuf csr_colf, col_cls;  // col_cls: one byte per column, its class
    int64_t col_class_cols[16] = {};
    // CSR: entry counts of the columns, left by feature extraction for the
    // plan (which frees them)
    gs::DevBuf col_counts;
    // CSR: entries inside their row tile's window, per candidate tile of 32,
    // 64, 128 and 256 rows with halo 0 / 1 (natural-order matrices without
    // long rows only; win_counted says whether they were counted)
    bool win_counted = false;
    int64_t win_entries[8] = {};
    // COO: rows with no entries (zeroed by the COO fixup launch), and the
    // entries with |col - row| < 4096 (which sets the number of rounds)
    int64_t n_empty_rows = 0;
    gs::DevBuf empty_rows;
    int64_t coo_local = 0;
    // COO: range boundaries (T + 1) and the split rows, {range q that begins
    // the row, row, later ranges the row runs into, 0}, per (T, per, S) the
    // SpMM calls have used
    struct CooRanges {
        gs::DevBuf bounds, split;
        int64_t n_split = 0;
    };
    std::map<std::tuple<int64_t, int64_t, int>, CooRanges> coo_ranges;

    // F-dependent workspace (partials / carries), grown on demand.
    gs::DevBuf work;

    uint64_t device_bytes = 0;

    // Work that reads the handle's arrays on a stream other than `stream`
    // (an SpMM, to_coo or an array copy): an event recorded after the last
    // such call, waited for before the arrays are freed (they are freed in
    // `stream` order, which does not cover other streams).
    hipEvent_t last_foreign = nullptr;

    gs_matrix_() = default;
    gs_matrix_(const gs_matrix_ &) = delete;
    gs_matrix_ &operator=(const gs_matrix_ &) = delete;
    ~gs_matrix_()
    {
        if (last_foreign) {
            (void)hipEventSynchronize(last_foreign);
            (void)hipEventDestroy(last_foreign);
        }
    }
};

namespace gs {

constexpr uint64_t kDefaultMaxBytes = 8ull << 30;
constexpr int kDefaultBsrBlock = 16;

// Rows longer than this go through the split (multi-workgroup) CSR path.
constexpr int kCsrLongRow = 128;
// Chunk length of the split CSR path.
constexpr int kCsrChunk = 128;
// Long rows up to this many entries take one workgroup on the vectorised
// path; longer ones are split across workgroups.
constexpr int kCsrWgRow = 1024;
// With many more long rows than resident workgroups, rows up to this many
// entries take one lane group each (summed in chunks of kCsrChunk).
constexpr int kCsrGroupRow = 2048;
// COO: range boundaries move to the next row start within at most kCooSnap
// entries, and a segment's running sum is folded every kCooFold entries;
// ranges hold at least kCooMinRange entries, and about kCooBandRange when
// they come in several rounds (so that with the move they stay within
// kCooFold).
constexpr int kCooSnap = 32;
constexpr int kCooFold = 128;
constexpr int kCooMinRange = 32;
constexpr int kCooBandRange = 48;
// BSR(16) hybrid plan: a block with at least this many entries (of 256)
// runs on the matrix cores, the entries of sparser blocks as a row list.
constexpr int kHybridDenseMin = 64;
// A 16x16 BSR block with at least this many stored columns counts as dense.
constexpr int kBsrDenseCols = 8;

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ----------------------------------------------------------- scan (gs_scan)

// Exclusive prefix sum of n int32 values (in may equal out).  out[n] is also
// written with the total when out_has_total.  Enqueued on s.
void exclusive_scan_i32(const int32_t *in, int32_t *out, int64_t n, bool out_has_total,
                        hipStream_t s);

// *out += part[0] + ... + part[G-1], enqueued on s: the second level of the
// reductions whose workgroups leave one partial each (one workgroup's atomics
// on a shared word are cheap, thousands queue up).
void add_partials_u64(const unsigned long long *part, int64_t G, unsigned long long *out, hipStream_t s);

// Stable LSD radix sort of n 64-bit keys on the 8-bit digits at `shifts`,
// least significant first, carrying a 32-bit payload that starts as the
// identity (the key's input position).  Ping-pongs between (ka, pa) and
// (kb, pb); *keys / *perm receive the buffers holding the result (*perm is
// null when no pass ran: the identity).  Enqueued on s.
void radix_sort_pairs(uint64_t *ka, uint64_t *kb, uint32_t *pa, uint32_t *pb, int64_t n,
                      const std::vector<int> &shifts, hipStream_t s, uint64_t **keys,
                      uint32_t **perm);
int bits_for(int64_t maxval);

// ------------------------------------------------------ build (gs_build)

struct CanonCOO {
    int64_t R = 0, C = 0, Z = 0;
    DevBuf row, col, val;     // canonical order (owned)
};

// Validates A and produces its canonical COO.  Throws Error on invalid input.
void canonicalize(const gs_coo &A, bool assume_canonical, hipStream_t s, CanonCOO &out);

// Builds a CSR handle from canonical COO (takes ownership of col/val).
// plan = false leaves the SpMM work plan to the first use of the handle
// (feature extraction reads only row_ptr / col).
gs_matrix_ *csr_from_canon(CanonCOO &&c, hipStream_t s, bool plan = true);

// Builds format fmt from a CSR handle (not consumed).
gs_matrix_ *convert_from_csr(const gs_matrix_ &csr, int fmt, int bsr_block, uint64_t max_bytes,
                             hipStream_t s, uint64_t *bytes_required);

// Canonical COO arrays of any handle into caller memory.
void to_coo(const gs_matrix_ &m, int32_t *row, int32_t *col, float *val, hipStream_t s);

// Builds a CSR handle from any handle (via its canonical COO).
gs_matrix_ *csr_from_any(const gs_matrix_ &m, hipStream_t s);

// Bytes a format would need for this CSR (from the features' aggregates).
uint64_t format_bytes(int fmt, int64_t R, int64_t C, int64_t Z, int64_t K, int64_t ND,
                      int64_t nb, int b);

// Counts distinct (row/b, col/b) blocks of a CSR matrix (device, synchronises).
int64_t count_blocks(const gs_matrix_ &csr, int b, hipStream_t s);
// Same, added to *total [dev] without waiting for the result.
void count_blocks_async(const gs_matrix_ &csr, int b, unsigned long long *total, hipStream_t s);

// --------------------------------------------------- features (gs_features)

// Keeps the column counts in csr.col_counts when csr has no work plan yet.
void features_from_csr(gs_matrix_ &csr, hipStream_t s, gs_features *out);
// Entry counts cc[0..C) of the columns of col[0..Z) (cc is cleared here).
void column_counts(const int32_t *col, int64_t C, int64_t Z, int32_t *cc, hipStream_t s);
// Diagonal occupancy bitmap of a CSR matrix: bit (col - row + R - 1) of
// bm[ceil((R+C-1)/32)] set for every entry; bm need not be cleared.
void diag_bitmap(const int32_t *rp, const int32_t *col, int64_t R, int64_t C, int64_t Z,
                 uint32_t *bm, hipStream_t s);

// ------------------------------------------------------- spmm (gs_spmm_*)

void spmm_csr(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s, const WorkArea *fixed = nullptr);
void spmm_coo(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s, const WorkArea *fixed = nullptr);
void spmm_ell(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s);
void spmm_dia(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s);
void spmm_bsr(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s);
void spmm_csc(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s, const WorkArea *fixed = nullptr);

// Plans built at conversion time for the CSR and COO kernels.
void plan_csr(gs_matrix_ &m, hipStream_t s);
// Entries inside their row tile's window for every candidate tile (T = 32,
// 64, 128, 256 rows, halo 0 / 1) of the matrix with CSR arrays rp, col, into
// m.win_entries (synchronises s).
void count_windows(gs_matrix_ &m, const int32_t *rp, const int32_t *col, hipStream_t s);
// The LDS-staged row tile for m at row_bytes of X per staged row: the
// counted candidate with the most in-window entries that fits the LDS budget,
// when at least 65% of the entries are inside and the matrix has at least two
// tiles per resident workgroup (false: no window).
bool pick_window(const gs_matrix_ &m, int64_t row_bytes, int &T, int &h);
void plan_coo(gs_matrix_ &m, const int32_t *row_ptr, hipStream_t s);

// Vectorised CSR path; returns false when F / alignment do not allow it.
bool spmm_csr_vec4(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                   hipStream_t s, const WorkArea *fixed = nullptr);

// Workgroups of 256 threads the device keeps resident at full occupancy
// (compute units x 8), queried once.
int resident_workgroups();
int compute_units();
// LDS bytes one workgroup may use (the device's limit), queried once.
int64_t max_lds_bytes();

// Vectorised ELL / DIA paths; false when F / alignment do not allow them.
bool spmm_ell_fast(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                   hipStream_t s);
bool spmm_dia_fast(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                   hipStream_t s);

// Hybrid plan of a 16x16 BSR handle from its CSR arrays (dense blocks on the
// matrix cores, the rest as rows); GS_BSR_HYBRID = off skips it.
void plan_bsr_hybrid(gs_matrix_ &m, const int32_t *rp, const int32_t *col, const float *val, hipStream_t s);

// 16x16-block BSR on the matrix cores; false when b != 16 or F % 16 != 0.
bool spmm_bsr16_mfma(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                     hipStream_t s);

// Makes sure m.work holds at least bytes (reallocating in stream order).
void ensure_work(gs_matrix_ &m, size_t bytes, hipStream_t s);

// Where an SpMM call takes its F-dependent workspace (partial sums of split
// rows, the CSC accumulator): the handle's own buffer, grown through the
// allocator on demand (fixed == nullptr), or a fixed buffer of cap bytes that
// is never grown.
struct WorkArea {
    void *p = nullptr;
    size_t cap = 0;
};

// A workspace of at least `bytes` for an SpMM on m: fixed->p when fixed is
// given (GS_ERR_UNSUPPORTED when bytes exceed fixed->cap), else m.work grown
// in stream order.
void *work_for(gs_matrix_ &m, const WorkArea *fixed, size_t bytes, hipStream_t s);

// Records that work reading m's arrays was enqueued on s (see
// gs_matrix_::last_foreign); nothing when s is m's own stream or is being
// captured into a graph (replays are ordered by the caller).
void note_use(gs_matrix_ &m, hipStream_t s);

// Argument checks of gs_spmm (throws Error) and the format dispatch.
void check_spmm_args(const gs_matrix_ *A, const float *X, int64_t ldx, const float *Y, int64_t ldy,
                     int64_t F);
void run_spmm(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s, const WorkArea *fixed = nullptr);

}  // namespace gs
