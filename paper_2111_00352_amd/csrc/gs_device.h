// Device-side helpers shared by the gfx950 kernels: XCD-aware workgroup
// remapping, wavefront reductions and vector access types.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gs {

constexpr int kWave = 64;  // CDNA wavefront width
// Every sequential fp32 sum runs at most this many terms before it is added
// into a running total (a row's rounding error then stays within 1e-5 of
// the sum of its absolute terms for rows of thousands of entries).
constexpr int kChainFold = 128;
constexpr int kXcds = 8;   // MI355X: 8 accelerator dies, each with its own L2

// The dispatcher hands consecutive workgroup ids to the XCDs round-robin.
// Remap so that XCD x processes one contiguous range of logical tiles: rows
// that are close in the matrix (and the X rows they share) then stay in one
// L2.  Bijective on [0, n).
__device__ __forceinline__ int64_t xcd_tile(int64_t bid, int64_t n)
{
    int64_t x = bid % kXcds, local = bid / kXcds;
    int64_t per = n / kXcds, rem = n % kXcds;
    return x * per + (x < rem ? x : rem) + local;
}

__device__ __forceinline__ int wave_min_i32(int v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        int w = __shfl_xor(v, o, kWave);
        v = w < v ? w : v;
    }
    return v;
}

__device__ __forceinline__ int wave_max_i32(int v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        int w = __shfl_xor(v, o, kWave);
        v = w > v ? w : v;
    }
    return v;
}

__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ int wave_sum_i32(int v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Workgroup-wide reductions over NT threads (a multiple of the wave width):
// every thread passes its value and receives the workgroup's result.  tmp
// holds NT / kWave values in LDS; the call ends with a barrier, so the next
// call may reuse tmp.
template <int NT>
__device__ __forceinline__ unsigned long long block_sum_u64(unsigned long long v, unsigned long long *tmp)
{
    v = wave_sum_u64(v);
    if (lane_id() == 0) tmp[threadIdx.x / kWave] = v;
    __syncthreads();
    unsigned long long t = 0;
    for (int w = 0; w < NT / kWave; w++) t += tmp[w];
    __syncthreads();
    return t;
}

template <int NT> __device__ __forceinline__ int block_max_i32(int v, int *tmp)
{
    v = wave_max_i32(v);
    if (lane_id() == 0) tmp[threadIdx.x / kWave] = v;
    __syncthreads();
    int t = tmp[0];
    for (int w = 1; w < NT / kWave; w++) t = tmp[w] > t ? tmp[w] : t;
    __syncthreads();
    return t;
}

template <int NT> __device__ __forceinline__ int block_min_i32(int v, int *tmp)
{
    v = wave_min_i32(v);
    if (lane_id() == 0) tmp[threadIdx.x / kWave] = v;
    __syncthreads();
    int t = tmp[0];
    for (int w = 1; w < NT / kWave; w++) t = tmp[w] < t ? tmp[w] : t;
    __syncthreads();
    return t;
}

// Exclusive prefix sum of one value per thread over the workgroup (NT
// threads); tmp holds NT / kWave ints.  Ends with a barrier.
template <int NT> __device__ __forceinline__ int block_exclusive_scan(int x, int *tmp)
{
    const int lane = lane_id(), w = threadIdx.x / kWave;
    int inc = x;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(inc, o, kWave);
        if (lane >= o) inc += y;
    }
    if (lane == kWave - 1) tmp[w] = inc;
    __syncthreads();
    int off = 0;
    for (int v = 0; v < w; v++) off += tmp[v];
    __syncthreads();
    return off + inc - x;
}

// fp32 vector of VEC elements with the alignment of its size.
template <int VEC> struct Vec;
template <> struct Vec<1> {
    float v[1];
};
template <> struct alignas(8) Vec<2> {
    float v[2];
};
template <> struct alignas(16) Vec<4> {
    float v[4];
};

template <int VEC>
__device__ __forceinline__ Vec<VEC> ld_vec(const float *p)
{
    return *reinterpret_cast<const Vec<VEC> *>(p);
}

template <int VEC>
__device__ __forceinline__ void st_vec(float *p, const Vec<VEC> &v)
{
    *reinterpret_cast<Vec<VEC> *>(p) = v;
}

// Streaming store: the output is not re-read by this kernel, keep it from
// displacing the gathered X rows in L2 / the MALL.
template <int VEC>
__device__ __forceinline__ void st_vec_stream(float *p, const Vec<VEC> &v)
{
#pragma unroll
    for (int i = 0; i < VEC; i++) __builtin_nontemporal_store(v.v[i], p + i);
}

template <class T>
__device__ __forceinline__ T ld_stream(const T *p)
{
    return __builtin_nontemporal_load(p);
}

}  // namespace gs
