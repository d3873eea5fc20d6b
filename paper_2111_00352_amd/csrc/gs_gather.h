// Shared inner loop of the vectorised SpMM kernels: a group of G lanes
// holds a batch of (column, value) pairs, one per lane, and gathers the
// corresponding X rows B at a time, each lane loading NQ float4 at columns
// c0 + 4*G*q (so one load instruction reads G*16 contiguous bytes of a row).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gs {

// Gathered X rows: plain cached loads (non-temporal loads measured slower:
// hub rows are reused from L2 and the MALL).
__device__ __forceinline__ float4 load_x4(const float *p)
{
    return *reinterpret_cast<const float4 *>(p);
}

// One batch of B entries j .. j+B-1 of the group's current index batch:
// B X-row loads issued back to back, then B fused multiply-adds.  MASKED
// batches may run past the last entry m: those slots gather a valid row
// (lane wrap) and are dropped by a select, so Inf/NaN in X cannot leak in.
template <int B, int NQ, int G, bool MASKED>
__device__ __forceinline__ void gather_batch(int cj, float vj, int j, int m,
                                             const float *__restrict__ X, int64_t ldx, int64_t c0,
                                             const bool *qok, float *acc)
{
    float4 x[B][NQ];
    float v[B];
#pragma unroll
    for (int u = 0; u < B; u++) {
        const int cu = __shfl(cj, j + u, G);
        v[u] = __shfl(vj, j + u, G);
        const float *xp = X + (int64_t)cu * ldx + c0;
#pragma unroll
        for (int q = 0; q < NQ; q++)
            x[u][q] = qok[q] ? load_x4(xp + 4 * G * q) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < B; u++) {
        const bool live = !MASKED || j + u < m;
#pragma unroll
        for (int q = 0; q < NQ; q++) {
            const float a0 = __builtin_fmaf(v[u], x[u][q].x, acc[4 * q + 0]);
            const float a1 = __builtin_fmaf(v[u], x[u][q].y, acc[4 * q + 1]);
            const float a2 = __builtin_fmaf(v[u], x[u][q].z, acc[4 * q + 2]);
            const float a3 = __builtin_fmaf(v[u], x[u][q].w, acc[4 * q + 3]);
            acc[4 * q + 0] = live ? a0 : acc[4 * q + 0];
            acc[4 * q + 1] = live ? a1 : acc[4 * q + 1];
            acc[4 * q + 2] = live ? a2 : acc[4 * q + 2];
            acc[4 * q + 3] = live ? a3 : acc[4 * q + 3];
        }
    }
}


// Stores NQ float4 of acc to row pointer p (columns c0 + 4*G*q), streaming.
template <int NQ, int G>
__device__ __forceinline__ void store_row_stream(float *p, const bool *qok, const float *acc)
{
#pragma unroll
    for (int q = 0; q < NQ; q++)
        if (qok[q]) {
#pragma unroll
            for (int i = 0; i < 4; i++) __builtin_nontemporal_store(acc[4 * q + i], p + 4 * G * q + i);
        }
}

template <int NQ, int G>
__device__ __forceinline__ void store_row(float *p, const bool *qok, const float *acc)
{
#pragma unroll
    for (int q = 0; q < NQ; q++)
        if (qok[q])
            *reinterpret_cast<float4 *>(p + 4 * G * q) =
                make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
}

}  // namespace gs
