// C ABI entry points for building, converting, inspecting and multiplying
// sparse matrices (the storage formats of Sec. 2.2, SpMM of Sec. 2.1,
// features of Sec. 4.4).  Argument checking and error translation happen
// here; the device work lives in gs_build / gs_features / gs_spmm.
#include <cstdint>
#include <cstring>

#include "gs_internal.h"

using namespace gs;

namespace gs {

void check_coo(const gs_coo *A)
{
    if (!A) fail(GS_ERR_INVALID_ARG, "null gs_coo");
    if (A->n_rows < 0 || A->n_cols < 0 || A->nnz < 0)
        fail(GS_ERR_INVALID_ARG, "negative matrix size");
    if (A->n_rows > INT32_MAX || A->n_cols > INT32_MAX || A->nnz > INT32_MAX)
        fail(GS_ERR_UNSUPPORTED, "matrix sizes must be below 2^31");
    if (A->nnz > 0 && (!A->row || !A->col || !A->val))
        fail(GS_ERR_INVALID_ARG, "null COO array with nnz > 0");
}

void check_spmm_args(const gs_matrix_ *A, const float *X, int64_t ldx, const float *Y, int64_t ldy,
                     int64_t F)
{
    if (!A) fail(GS_ERR_INVALID_ARG, "null matrix handle");
    if (F <= 0) fail(GS_ERR_INVALID_ARG, "F must be positive (got %lld)", (long long)F);
    if (F > (int64_t(1) << 24)) fail(GS_ERR_UNSUPPORTED, "F = %lld exceeds 2^24 columns", (long long)F);
    if (ldx < F || ldy < F) fail(GS_ERR_INVALID_ARG, "leading dimensions must be >= F");
    // each operand spans (rows - 1) * ld + F floats; the overlap test below
    // needs that in bytes without overflow
    auto fits = [F](int64_t rows, int64_t ld) {
        return rows <= 1 || (rows - 1) <= (INT64_MAX / 4 - F) / ld;
    };
    if (!fits(A->C, ldx) || !fits(A->R, ldy)) fail(GS_ERR_INVALID_ARG, "leading dimension too large");
    if ((A->C > 0 && !X) || (A->R > 0 && !Y)) fail(GS_ERR_INVALID_ARG, "null X or Y");
    if (A->C > 0 && A->R > 0) {
        const uintptr_t x0 = (uintptr_t)X, x1 = x0 + (uintptr_t)(((A->C - 1) * ldx + F) * 4);
        const uintptr_t y0 = (uintptr_t)Y, y1 = y0 + (uintptr_t)(((A->R - 1) * ldy + F) * 4);
        if (x0 < y1 && y0 < x1) fail(GS_ERR_INVALID_ARG, "X and Y overlap");
    }
}

gs_build_opts resolve_opts(const gs_build_opts *o)
{
    gs_build_opts r = {kDefaultBsrBlock, 0, kDefaultMaxBytes};
    if (o) {
        r = *o;
        if (r.bsr_block == 0) r.bsr_block = kDefaultBsrBlock;
        if (r.max_bytes == 0) r.max_bytes = kDefaultMaxBytes;
    }
    if (r.bsr_block < 1 || r.bsr_block > 64)
        fail(GS_ERR_INVALID_ARG, "bsr_block %d outside 1..64", r.bsr_block);
    return r;
}

gs_matrix_ *build_csr(const gs_coo *A, const gs_build_opts &o, hipStream_t s, bool plan)
{
    CanonCOO c;
    canonicalize(*A, o.assume_canonical != 0, s, c);
    return csr_from_canon(std::move(c), s, plan);
}

void run_spmm(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s, const WorkArea *fixed)
{
    if (m.R == 0) return;
    switch (m.fmt) {
    case GS_CSR: spmm_csr(m, X, ldx, Y, ldy, F, s, fixed); break;
    case GS_COO: spmm_coo(m, X, ldx, Y, ldy, F, s, fixed); break;
    case GS_ELL: spmm_ell(m, X, ldx, Y, ldy, F, s); break;
    case GS_DIA: spmm_dia(m, X, ldx, Y, ldy, F, s); break;
    case GS_BSR: spmm_bsr(m, X, ldx, Y, ldy, F, s); break;
    case GS_CSC: spmm_csc(m, X, ldx, Y, ldy, F, s, fixed); break;
    default: fail(GS_ERR_INVALID_ARG, "corrupt matrix handle");
    }
    note_use(m, s);
}

}  // namespace gs

extern "C" {

int gs_build_format(const gs_coo *A, int fmt, const gs_build_opts *opts, gs_stream stream,
                    gs_matrix *out, uint64_t *bytes_required)
{
    if (out) *out = nullptr;
    return guarded([&] {
        if (!out) fail(GS_ERR_INVALID_ARG, "null output handle");
        if (fmt < 0 || fmt >= GS_NUM_FORMATS) fail(GS_ERR_INVALID_ARG, "unknown format %d", fmt);
        check_coo(A);
        const gs_build_opts o = resolve_opts(opts);
        hipStream_t s = (hipStream_t)stream;
        gs_matrix_ *csr = build_csr(A, o, s, fmt == GS_CSR);
        if (fmt == GS_CSR) {
            if (bytes_required) *bytes_required = csr->device_bytes;
            *out = csr;
            return;
        }
        try {
            *out = convert_from_csr(*csr, fmt, o.bsr_block, o.max_bytes, s, bytes_required);
        } catch (...) {
            delete csr;
            throw;
        }
        delete csr;
    });
}

int gs_convert(gs_matrix A, int fmt, const gs_build_opts *opts, gs_stream stream, gs_matrix *out,
               uint64_t *bytes_required)
{
    if (out) *out = nullptr;
    return guarded([&] {
        if (!out || !A) fail(GS_ERR_INVALID_ARG, "null handle");
        if (fmt < 0 || fmt >= GS_NUM_FORMATS) fail(GS_ERR_INVALID_ARG, "unknown format %d", fmt);
        const gs_build_opts o = resolve_opts(opts);
        hipStream_t s = (hipStream_t)stream;
        if (A->fmt == GS_CSR) {
            *out = convert_from_csr(*A, fmt, o.bsr_block, o.max_bytes, s, bytes_required);
            return;
        }
        gs_matrix_ *csr = csr_from_any(*A, s);
        try {
            *out = convert_from_csr(*csr, fmt, o.bsr_block, o.max_bytes, s, bytes_required);
        } catch (...) {
            delete csr;
            throw;
        }
        delete csr;
    });
}

int gs_spmm(gs_matrix A, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
            gs_stream stream)
{
    return guarded([&] {
        check_spmm_args(A, X, ldx, Y, ldy, F);
        run_spmm(*A, X, ldx, Y, ldy, F, (hipStream_t)stream);
    });
}

int gs_to_coo(gs_matrix A, int32_t *row, int32_t *col, float *val, gs_stream stream)
{
    return guarded([&] {
        if (!A) fail(GS_ERR_INVALID_ARG, "null matrix handle");
        if (A->Z > 0 && (!row || !col || !val)) fail(GS_ERR_INVALID_ARG, "null output array");
        to_coo(*A, row, col, val, (hipStream_t)stream);
        note_use(*A, (hipStream_t)stream);
    });
}

int gs_extract_features(const gs_coo *A, const gs_build_opts *opts, gs_stream stream,
                        gs_features *out)
{
    return guarded([&] {
        if (!out) fail(GS_ERR_INVALID_ARG, "null output");
        check_coo(A);
        const gs_build_opts o = resolve_opts(opts);
        hipStream_t s = (hipStream_t)stream;
        gs_matrix_ *csr = build_csr(A, o, s, false);
        try {
            features_from_csr(*csr, s, out);
        } catch (...) {
            delete csr;
            throw;
        }
        delete csr;
    });
}

int gs_matrix_features(gs_matrix A, gs_stream stream, gs_features *out)
{
    return guarded([&] {
        if (!A || !out) fail(GS_ERR_INVALID_ARG, "null argument");
        hipStream_t s = (hipStream_t)stream;
        if (A->fmt == GS_CSR) {
            features_from_csr(*A, s, out);
            return;
        }
        gs_matrix_ *csr = csr_from_any(*A, s);
        try {
            features_from_csr(*csr, s, out);
        } catch (...) {
            delete csr;
            throw;
        }
        delete csr;
    });
}

}  // extern "C"
