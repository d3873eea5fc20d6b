// Device exclusive prefix sum over int32 (reduce -> scan of tile sums ->
// scan of tiles), used by the format builders for row pointers, block
// pointers, diagonal numbering and output positions.
#include "gs_device.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kSB = 256;         // threads per block
constexpr int kSI = 8;           // items per thread
constexpr int kST = kSB * kSI;   // items per tile

// Exclusive scan of one value per thread across the block; returns the
// block total through *total.
__device__ int block_exclusive_scan(int v, int *total)
{
    __shared__ int wsum[kSB / kWave];
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    int x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) wsum[w] = x;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < kSB / kWave; i++) {
        if (i < w) before += wsum[i];
        all += wsum[i];
    }
    __syncthreads();
    *total = all;
    return before + x - v;
}

__global__ __launch_bounds__(kSB) void k_tile_sums(const int32_t *__restrict__ in, int64_t n,
                                                   int32_t *__restrict__ sums)
{
    const int64_t base = (int64_t)blockIdx.x * kST;
    int s = 0;
#pragma unroll
    for (int i = 0; i < kSI; i++) {
        int64_t k = base + (int64_t)i * kSB + threadIdx.x;
        if (k < n) s += in[k];
    }
    int total;
    block_exclusive_scan(s, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kSB) void k_scan_tiles(const int32_t *in, int32_t *out, int64_t n,
                                                    const int32_t *__restrict__ tile_off,
                                                    int write_total)
{
    const int64_t base = (int64_t)blockIdx.x * kST + (int64_t)threadIdx.x * kSI;
    int v[kSI];
    int s = 0;
#pragma unroll
    for (int i = 0; i < kSI; i++) {
        v[i] = (base + i < n) ? in[base + i] : 0;
        s += v[i];
    }
    int total;
    int run = block_exclusive_scan(s, &total) + (tile_off ? tile_off[blockIdx.x] : 0);
#pragma unroll
    for (int i = 0; i < kSI; i++) {
        if (base + i < n) {
            out[base + i] = run;
            if (write_total && base + i == n - 1) out[n] = run + v[i];
        }
        run += v[i];
    }
}

// *out += part[0] + ... + part[G-1] (one workgroup).
__global__ __launch_bounds__(kSB) void k_add_partials(const unsigned long long *__restrict__ part, int64_t G,
                                                      unsigned long long *__restrict__ out)
{
    __shared__ unsigned long long t64[kSB / kWave];
    unsigned long long t = 0;
    for (int64_t g = threadIdx.x; g < G; g += kSB) t += part[g];
    t = block_sum_u64<kSB>(t, t64);
    if (threadIdx.x == 0) *out += t;
}

}  // namespace

void exclusive_scan_i32(const int32_t *in, int32_t *out, int64_t n, bool out_has_total,
                        hipStream_t s)
{
    if (n <= 0) {
        if (out_has_total) GS_HIP(hipMemsetAsync(out, 0, sizeof(int32_t), s));
        return;
    }
    const int64_t tiles = ceil_div(n, kST);
    if (tiles == 1) {
        k_scan_tiles<<<1, kSB, 0, s>>>(in, out, n, nullptr, out_has_total ? 1 : 0);
        GS_HIP(hipGetLastError());
        return;
    }
    DevBuf sums;
    sums.alloc((size_t)tiles * sizeof(int32_t), s);
    k_tile_sums<<<(unsigned)tiles, kSB, 0, s>>>(in, n, sums.as<int32_t>());
    GS_HIP(hipGetLastError());
    exclusive_scan_i32(sums.as<int32_t>(), sums.as<int32_t>(), tiles, false, s);
    k_scan_tiles<<<(unsigned)tiles, kSB, 0, s>>>(in, out, n, sums.as<int32_t>(),
                                                  out_has_total ? 1 : 0);
    GS_HIP(hipGetLastError());
}

void add_partials_u64(const unsigned long long *part, int64_t G, unsigned long long *out, hipStream_t s)
{
    if (G <= 0) return;
    k_add_partials<<<1, kSB, 0, s>>>(part, G, out);
    GS_HIP(hipGetLastError());
}

}  // namespace gs
