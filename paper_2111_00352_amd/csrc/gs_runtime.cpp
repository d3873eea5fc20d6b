// Error reporting, device allocation and matrix-handle plumbing of the C ABI.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>

#include "gs_internal.h"

namespace gs {

static thread_local char g_err[512] = "no error";

void set_error(const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
}

void fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    throw Error{code};
}

void hip_check(hipError_t e, const char *what)
{
    if (e != hipSuccess) fail(GS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

static gs_allocator g_alloc = {nullptr, nullptr, nullptr};

void *dev_alloc(size_t bytes, hipStream_t s, gs_allocator *used)
{
    *used = g_alloc;
    if (bytes == 0) return nullptr;
    void *p = nullptr;
    if (g_alloc.alloc) {
        p = g_alloc.alloc(bytes, s, g_alloc.ctx);
        if (!p) fail(GS_ERR_OOM, "device allocator returned NULL for %zu bytes", bytes);
        if (reinterpret_cast<uintptr_t>(p) & 255) {
            g_alloc.free(p, s, g_alloc.ctx);
            fail(GS_ERR_INVALID_ARG, "device allocator returned memory not aligned to 256 bytes");
        }
    } else {
        hipError_t e = hipMalloc(&p, bytes);
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            fail(GS_ERR_OOM, "hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
        }
    }
    return p;
}

void dev_free(void *p, hipStream_t s, const gs_allocator &used)
{
    if (!p) return;
    if (used.free) {
        used.free(p, s, used.ctx);  // stream-ordered by contract
    } else {
        // the library frees temporaries while work using them may still be
        // queued on s
        (void)hipStreamSynchronize(s);
        (void)hipFree(p);
    }
}

void ensure_work(gs_matrix_ &m, size_t bytes, hipStream_t s)
{
    if (m.work.bytes >= bytes) return;
    // The old workspace may still be read by work queued on its stream.
    if (m.work.p) GS_HIP(hipStreamSynchronize(m.work.s));
    m.work.alloc(bytes, s);
}

void *work_for(gs_matrix_ &m, const WorkArea *fixed, size_t bytes, hipStream_t s)
{
    if (fixed) {
        if (bytes > fixed->cap)
            fail(GS_ERR_UNSUPPORTED, "this SpMM needs %zu bytes of workspace, above the fixed %zu-byte scratch",
                 bytes, fixed->cap);
        return fixed->p;
    }
    ensure_work(m, bytes, s);
    return m.work.p;
}

void note_use(gs_matrix_ &m, hipStream_t s)
{
    if (s == m.stream) return;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess) {  // e.g. the legacy stream during a capture
        (void)hipGetLastError();
        return;
    }
    if (cs != hipStreamCaptureStatusNone) return;
    if (!m.last_foreign) GS_HIP(hipEventCreateWithFlags(&m.last_foreign, hipEventDisableTiming));
    GS_HIP(hipEventRecord(m.last_foreign, s));
}

// Device properties, read once (thread-safe static initialisation; a failed
// query throws and is retried on the next call).
int compute_units()
{
    static const int n = [] {
        int dev = 0, cus = 0;
        GS_HIP(hipGetDevice(&dev));
        GS_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
        return cus > 0 ? cus : 256;
    }();
    return n;
}

int resident_workgroups() { return compute_units() * 8; }

int64_t max_lds_bytes()
{
    static const int64_t n = [] {
        int dev = 0, v = 0;
        GS_HIP(hipGetDevice(&dev));
        GS_HIP(hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev));
        return (int64_t)(v > 0 ? v : 65536);
    }();
    return n;
}

}  // namespace gs

using namespace gs;

extern "C" {

const char *gs_last_error(void) { return g_err; }

int gs_abi_version(void) { return GS_ABI_VERSION; }

int gs_set_allocator(const gs_allocator *a)
{
    if (a && ((a->alloc == nullptr) != (a->free == nullptr))) {
        set_error("gs_set_allocator: alloc and free must both be set or both be NULL");
        return GS_ERR_INVALID_ARG;
    }
    if (a)
        g_alloc = *a;
    else
        g_alloc = gs_allocator{nullptr, nullptr, nullptr};
    return GS_OK;
}

void gs_destroy(gs_matrix A) { delete A; }

int gs_get_info(gs_matrix A, gs_matrix_info *info)
{
    if (!A || !info) {
        set_error("gs_get_info: null argument");
        return GS_ERR_INVALID_ARG;
    }
    info->format = A->fmt;
    info->bsr_block = A->fmt == GS_BSR ? A->b : 0;
    info->n_rows = A->R;
    info->n_cols = A->C;
    info->nnz = A->Z;
    info->param = A->fmt == GS_ELL ? A->K : A->fmt == GS_DIA ? A->ND : A->fmt == GS_BSR ? A->nb : 0;
    info->device_bytes = A->device_bytes;
    return GS_OK;
}

int gs_get_array(gs_matrix A, int which, const void **dev_ptr, uint64_t *bytes)
{
    if (!A || !dev_ptr || !bytes || which < 0 || which > 2) {
        set_error("gs_get_array: bad argument");
        return GS_ERR_INVALID_ARG;
    }
    const DevBuf *b = nullptr;
    switch (A->fmt) {
    case GS_COO: b = which == 0 ? &A->row : which == 1 ? &A->col : &A->val; break;
    case GS_CSR:
    case GS_CSC: b = which == 0 ? &A->row_ptr : which == 1 ? &A->col : &A->val; break;
    case GS_ELL:
        if (which == 2) {
            set_error("gs_get_array: ELL has arrays 0 (ell_col) and 1 (ell_val)");
            return GS_ERR_INVALID_ARG;
        }
        b = which == 0 ? &A->ell_col : &A->ell_val;
        break;
    case GS_DIA:
        if (which == 2) {
            set_error("gs_get_array: DIA has arrays 0 (offsets) and 1 (data)");
            return GS_ERR_INVALID_ARG;
        }
        b = which == 0 ? &A->offsets : &A->dia;
        break;
    case GS_BSR: b = which == 0 ? &A->bptr : which == 1 ? &A->bcol : &A->bval; break;
    default: set_error("gs_get_array: corrupt handle"); return GS_ERR_INVALID_ARG;
    }
    *dev_ptr = b->p;
    *bytes = b->bytes;
    return GS_OK;
}

int gs_copy_array(gs_matrix A, int which, void *dst, uint64_t dst_bytes, gs_stream s)
{
    const void *src = nullptr;
    uint64_t bytes = 0;
    int rc = gs_get_array(A, which, &src, &bytes);
    if (rc != GS_OK) return rc;
    if (bytes > dst_bytes || (bytes && !dst)) {
        set_error("gs_copy_array: destination too small or null");
        return GS_ERR_INVALID_ARG;
    }
    return guarded([&] {
        if (bytes) {
            GS_HIP(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, (hipStream_t)s));
            note_use(*A, (hipStream_t)s);
        }
    });
}

}  // extern "C"
