// Shared inner loop of the vectorised SpMM kernels: a group of G lanes
// holds a batch of (column, value) pairs, one per lane, and gathers the
// corresponding X rows B at a time, each lane loading NQ float4 at columns
// c0 + 4*G*q (so one load instruction reads G*16 contiguous bytes of a row).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gs {

// Gathered X rows: plain cached loads (non-temporal loads for every row
// measured slower: hub rows are reused from L2 and the MALL).
__device__ __forceinline__ float4 load_x4(const float *p)
{
    return *reinterpret_cast<const float4 *>(p);
}

// Non-temporal gather of a row that few entries reference: its lines are
// inserted for early eviction, so they do not push the rows of often
// referenced columns out of L2.
__device__ __forceinline__ float4 load_x4_nt(const float *p)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    const f4 v = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}

// Column words with a reference class: bits 27..30 hold the class of the
// column (bit length of its entry count, at most 15), bits 0..26 the column.
constexpr int kColClassShift = 27;
constexpr int kColMask = (1 << kColClassShift) - 1;

// One batch of B entries j .. j+B-1 of the group's current index batch:
// B X-row loads issued back to back, then B fused multiply-adds.  MASKED
// batches may run past the last entry m: those slots gather a valid row
// (lane wrap) and are dropped by a select, so Inf/NaN in X cannot leak in.
//
// CLS: cj holds class-tagged column words; rows of columns whose class is
// below hot_cls are gathered non-temporally.
template <int B, int NQ, int G, bool MASKED, bool CLS = false, bool FENCE = false>
__device__ __forceinline__ void gather_batch(int cj, float vj, int j, int m,
                                             const float *__restrict__ X, int64_t ldx, int64_t c0,
                                             const bool *qok, float *acc, int hot_cls = 0)
{
    float4 x[B][NQ];
    float v[B];
#pragma unroll
    for (int u = 0; u < B; u++) {
        const int cw = __shfl(cj, j + u, G);
        const int cu = CLS ? (cw & kColMask) : cw;
        v[u] = __shfl(vj, j + u, G);
        const float *xp = X + (int64_t)cu * ldx + c0;
        if (CLS && (cw >> kColClassShift) < hot_cls) {
#pragma unroll
            for (int q = 0; q < NQ; q++)
                x[u][q] = qok[q] ? load_x4_nt(xp + 4 * G * q) : make_float4(0.f, 0.f, 0.f, 0.f);
        } else {
#pragma unroll
            for (int q = 0; q < NQ; q++)
                x[u][q] = qok[q] ? load_x4(xp + 4 * G * q) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    // FENCE: every load of the batch is issued before the first use.  Where
    // the scheduler aims at a higher occupancy it may otherwise sink each
    // load next to its use, one round trip per X row (seen in the ELL kernel
    // with chain folds: 50 VGPRs and twice the time on a power-law matrix).
    if constexpr (FENCE) __builtin_amdgcn_sched_barrier(0);
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


// One batch of B entries j .. j+B-1 of the group's index batch in a row
// tile whose X rows [w0, w1) are staged in LDS (xs, G*NQ float4 per row, the
// lane's float4 at lane + G*q): in-window rows are read from LDS, the others
// from global memory.  Slots past m gather a valid row and are dropped by a
// select.
template <int B, int NQ, int G>
__device__ __forceinline__ void window_batch(int cj, float vj, int j, int m, const float4 *xs, int64_t w0,
                                             int64_t w1, int lane, const float *__restrict__ X, int64_t ldx,
                                             int64_t c0, const bool *qok, float *acc)
{
    constexpr int RW = G * NQ;
    float4 x[B][NQ];
    float v[B];
#pragma unroll
    for (int u = 0; u < B; u++) {
        const int cu = __shfl(cj, j + u, G);
        v[u] = __shfl(vj, j + u, G);
        if (cu >= w0 && cu < w1) {
            const float4 *xr = xs + (int64_t)(cu - w0) * RW + lane;
#pragma unroll
            for (int q = 0; q < NQ; q++) x[u][q] = xr[q * G];
        } else {
            const float *xp = X + (int64_t)cu * ldx + c0;
#pragma unroll
            for (int q = 0; q < NQ; q++)
                x[u][q] = qok[q] ? load_x4(xp + 4 * G * q) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
#pragma unroll
    for (int u = 0; u < B; u++) {
        const bool live = j + u < m;
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
