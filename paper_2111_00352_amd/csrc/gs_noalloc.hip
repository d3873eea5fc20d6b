// The allocation-free SpMM entry point: gs_spmm whose F-dependent workspace
// (partial sums of split CSR rows, the CSC fp64 accumulator) lives in a fixed
// device array instead of the handle's own buffer, so that the call never
// reaches the allocator.
//
// The array is a file-scope device variable.  Its name is only a host-side
// stand-in for the device copy, so host code never passes it to a kernel:
// each device's address is fetched once with hipGetSymbolAddress (with that
// device current) and kept per device.
#include <mutex>
#include <vector>

#include "gs_internal.h"

static __device__ __align__(256) unsigned char scratch[GS_NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex g_mu;
std::vector<void *> g_scratch;  // per device ordinal: address of that device's array

// Address of the current device's copy of `scratch`, looked up on the first
// call made with that device current.
void *device_scratch()
{
    int dev = 0;
    GS_HIP(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lock(g_mu);
    if ((size_t)dev >= g_scratch.size()) g_scratch.resize((size_t)dev + 1, nullptr);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            gs::fail(GS_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        g_scratch[dev] = p;
    }
    return g_scratch[dev];
}

}  // namespace

extern "C" int gs_spmm_noalloc(gs_matrix A, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                               gs_stream stream)
{
    return gs::guarded([&] {
        gs::check_spmm_args(A, X, ldx, Y, ldy, F);
        if (A->fmt == GS_COO) gs::fail(GS_ERR_UNSUPPORTED, "gs_spmm_noalloc: COO handles are not supported");
        const gs::WorkArea w{device_scratch(), (size_t)GS_NOALLOC_SCRATCH_BYTES};
        gs::run_spmm(*A, X, ldx, Y, ldy, F, (hipStream_t)stream, &w);
    });
}
