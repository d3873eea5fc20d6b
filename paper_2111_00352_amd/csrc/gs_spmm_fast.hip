// Vectorised ELL and DIA SpMM (F a multiple of 4, 16-byte aligned operands).
//
// Same lane layout as the CSR kernel: a group of G lanes owns one output
// row, lane l holding float4 q at column c0 + 4*G*q (CPL = 4*NQ columns per
// lane), and the persistent grid walks row tiles in natural order, so
// neighbouring rows -- which share X rows in banded / clustered matrices --
// run at the same time on the same XCD.
//
// ELL: slot k of row i lives at k*R + i; the group loads G slots at once
// (one per lane), the stored ones form a prefix (rows are packed to the
// front), and their X rows are gathered B at a time.
//
// DIA: the group loads the values and offsets of G diagonals at once (one
// per lane), then gathers X[i + off_d] for the stored ones (value != 0 and
// column inside the matrix) B at a time; padding slots are skipped.
#include <algorithm>
#include <cstdlib>

#include "gs_device.h"
#include "gs_gather.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kBlock = 256;

// FOLD: rows may hold more than kChainFold slots; their running sum is then
// added into a total every kChainFold slots (compiled out otherwise).
template <int CPL, int G, bool FULL, bool FOLD>
__global__ __launch_bounds__(kBlock) void k_ell_fast(int64_t R, int64_t K,
                                                     const int32_t *__restrict__ ec,
                                                     const float *__restrict__ ev,
                                                     const float *__restrict__ X, int64_t ldx,
                                                     float *__restrict__ Y, int64_t ldy, int64_t F)
{
    constexpr int GPB = kBlock / G;
    constexpr int NQ = CPL / 4;
    constexpr int U0 = 32 / CPL > 0 ? 32 / CPL : 1;
    constexpr int U = U0 < G ? U0 : G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int gbase = (threadIdx.x % kWave) / G * G;
    const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
    const int64_t c0 = (int64_t)blockIdx.y * (G * CPL) + (int64_t)lane * 4;
    bool qok[NQ];
#pragma unroll
    for (int q = 0; q < NQ; q++) qok[q] = FULL || (c0 + 4 * G * q < F);
    const int64_t tiles = (R + GPB - 1) / GPB;
    for (int64_t tile = xcd_tile(blockIdx.x, gridDim.x); tile < tiles; tile += gridDim.x) {
        const int64_t row = tile * GPB + g;
        if (row >= R) break;
        float acc[CPL], tot[FOLD ? CPL : 1];
#pragma unroll
        for (int i = 0; i < CPL; i++) acc[i] = 0.0f;
        if constexpr (FOLD) {
#pragma unroll
            for (int i = 0; i < CPL; i++) tot[i] = 0.0f;
        }
        // chains of kChainFold slots (one chain of K without FOLD; kChainFold
        // is a multiple of G), each added into the total when it ends
        const int64_t span = FOLD ? kChainFold : K;
        bool more = true;
        for (int64_t kc = 0; kc < K && more; kc += span) {
          const int64_t kend = kc + span < K ? kc + span : K;
          for (int64_t kb = kc; kb < kend; kb += G) {
            int cj = -1;
            float vj = 0.0f;
            if (kb + lane < K) {
                cj = ld_stream(ec + (kb + lane) * R + row);
                vj = ld_stream(ev + (kb + lane) * R + row);
            }
            const int m = __popcll((__ballot(cj >= 0) >> gbase) & gmask);
            if (cj < 0) cj = 0;  // padding lanes gather row 0 and are masked
            int j = 0;
            for (; j + U <= m; j += U) gather_batch<U, NQ, G, false, false, FOLD>(cj, vj, j, m, X, ldx, c0, qok, acc);
            if (j < m) {
                if (U > 1 && m - j <= U / 2)
                    gather_batch<(U > 1 ? U / 2 : 1), NQ, G, true, false, FOLD>(cj, vj, j, m, X, ldx, c0, qok, acc);
                else
                    gather_batch<U, NQ, G, true, false, FOLD>(cj, vj, j, m, X, ldx, c0, qok, acc);
            }
            if (m < G) {  // padding reached: the row has no more slots
                more = false;
                break;
            }
          }
          if constexpr (FOLD) {
#pragma unroll
            for (int i = 0; i < CPL; i++) {
                tot[i] += acc[i];
                acc[i] = 0.0f;
            }
          }
        }
        if constexpr (FOLD) {
#pragma unroll
            for (int i = 0; i < CPL; i++) acc[i] = tot[i];
        }
        store_row_stream<NQ, G>(Y + row * ldy + c0, qok, acc);
    }
}

// ELL with the X rows of each row tile staged in LDS, for natural-order
// matrices whose entries mostly stay near the diagonal (at most kChainFold
// slots per row: one chain).  A workgroup takes T consecutive rows [r0, r1),
// copies the X rows [r0 - halo, r1 + halo) of its column slice into LDS with
// coalesced loads, and its groups run the rows as k_ell_fast does, reading
// in-window columns from LDS and the others from global memory.
template <int CPL, int G, bool FULL>
__global__ __launch_bounds__(kBlock) void k_ell_window(int64_t R, int64_t C, int64_t K,
                                                       const int32_t *__restrict__ ec,
                                                       const float *__restrict__ ev,
                                                       const float *__restrict__ X, int64_t ldx,
                                                       float *__restrict__ Y, int64_t ldy, int64_t F, int T,
                                                       int halo, int64_t ntiles)
{
    constexpr int GPB = kBlock / G;
    constexpr int NQ = CPL / 4;
    constexpr int RW = G * NQ;  // float4 per staged row
    constexpr int B0 = 32 / CPL > 0 ? 32 / CPL : 1;
    constexpr int B = B0 < G ? B0 : G;  // X rows in flight per batch
    extern __shared__ float4 xs[];
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int gbase = (threadIdx.x % kWave) / G * G;
    const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
    const int64_t cbase = (int64_t)blockIdx.y * (G * CPL);
    const int64_t c0 = cbase + (int64_t)lane * 4;
    bool qok[NQ];
#pragma unroll
    for (int q = 0; q < NQ; q++) qok[q] = FULL || (c0 + 4 * G * q < F);

    for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const int64_t r0 = t * T, r1 = r0 + T < R ? r0 + T : R;
        const int64_t w0 = r0 - halo > 0 ? r0 - halo : 0;
        const int64_t w1 = r1 + halo < C ? r1 + halo : C;
        const int W = w1 > w0 ? (int)(w1 - w0) : 0;
        __syncthreads();  // the previous tile's rows are done with xs
        for (int idx = threadIdx.x; idx < W * RW; idx += kBlock) {
            const int wr = idx / RW, j = idx - wr * RW;
            const int64_t cc = cbase + 4 * j;
            xs[idx] = (FULL || cc < F) ? load_x4(X + (w0 + wr) * ldx + cc) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        __syncthreads();
        for (int64_t r = r0 + g; r < r1; r += GPB) {
            float acc[CPL];
#pragma unroll
            for (int i = 0; i < CPL; i++) acc[i] = 0.0f;
            for (int64_t kb = 0; kb < K; kb += G) {
                int cj = -1;
                float vj = 0.0f;
                if (kb + lane < K) {
                    cj = ld_stream(ec + (kb + lane) * R + r);
                    vj = ld_stream(ev + (kb + lane) * R + r);
                }
                const int m = __popcll((__ballot(cj >= 0) >> gbase) & gmask);
                if (cj < 0) cj = 0;  // padding lanes gather row 0 and are masked
                for (int j = 0; j < m; j += B)
                    window_batch<B, NQ, G>(cj, vj, j, m, xs, w0, w1, lane, X, ldx, c0, qok, acc);
                if (m < G) break;
            }
            store_row_stream<NQ, G>(Y + r * ldy + c0, qok, acc);
        }
    }
}

// FOLD: more than kChainFold diagonals (the running sum of a row is added
// into a total every kChainFold diagonals; compiled out otherwise).
template <int CPL, int G, bool FULL, bool FOLD>
__global__ __launch_bounds__(kBlock) void k_dia_fast(int64_t R, int64_t C, int64_t ND,
                                                     const int32_t *__restrict__ offsets,
                                                     const float *__restrict__ data,
                                                     const float *__restrict__ X, int64_t ldx,
                                                     float *__restrict__ Y, int64_t ldy, int64_t F)
{
    constexpr int GPB = kBlock / G;
    constexpr int NQ = CPL / 4;
    constexpr int U0 = 32 / CPL > 0 ? 32 / CPL : 1;
    constexpr int U = U0 < G ? U0 : G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int gbase = (threadIdx.x % kWave) / G * G;
    const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
    const int64_t c0 = (int64_t)blockIdx.y * (G * CPL) + (int64_t)lane * 4;
    bool qok[NQ];
#pragma unroll
    for (int q = 0; q < NQ; q++) qok[q] = FULL || (c0 + 4 * G * q < F);
    const int64_t tiles = (R + GPB - 1) / GPB;
    for (int64_t tile = xcd_tile(blockIdx.x, gridDim.x); tile < tiles; tile += gridDim.x) {
        const int64_t row = tile * GPB + g;
        if (row >= R) break;
        float acc[CPL], tot[FOLD ? CPL : 1];
#pragma unroll
        for (int i = 0; i < CPL; i++) acc[i] = 0.0f;
        if constexpr (FOLD) {
#pragma unroll
            for (int i = 0; i < CPL; i++) tot[i] = 0.0f;
        }
        for (int64_t db = 0; db < ND; db += G) {
            if (FOLD && db > 0 && db % kChainFold == 0) {  // fold the running chain every kChainFold diagonals
#pragma unroll
                for (int i = 0; i < CPL; i++) {
                    tot[i] += acc[i];
                    acc[i] = 0.0f;
                }
            }
            int cj = 0;
            float vj = 0.0f;
            bool ok = false;
            if (db + lane < ND) {
                vj = ld_stream(data + (db + lane) * R + row);
                const int64_t j = row + offsets[db + lane];
                ok = vj != 0.0f && j >= 0 && j < C;
                cj = ok ? (int)j : 0;
            }
            // compact the stored diagonals to the front of the group: lane t
            // takes the t-th set bit of the group's "stored" mask
            const uint64_t live = (__ballot(ok) >> gbase) & gmask;
            const int m = __popcll(live);
            uint64_t bits = live;
            for (int t = 0; t < lane && bits; t++) bits &= bits - 1;
            const int pick = bits ? __ffsll((unsigned long long)bits) - 1 : 0;
            const int cc = __shfl(cj, pick, G);
            const float vv = __shfl(vj, pick, G);
            int j = 0;
            for (; j + U <= m; j += U) gather_batch<U, NQ, G, false, false, FOLD>(cc, vv, j, m, X, ldx, c0, qok, acc);
            if (j < m) {
                if (U > 1 && m - j <= U / 2)
                    gather_batch<(U > 1 ? U / 2 : 1), NQ, G, true, false, FOLD>(cc, vv, j, m, X, ldx, c0, qok, acc);
                else
                    gather_batch<U, NQ, G, true, false, FOLD>(cc, vv, j, m, X, ldx, c0, qok, acc);
            }
        }
        if constexpr (FOLD) {
#pragma unroll
            for (int i = 0; i < CPL; i++) acc[i] += tot[i];
        }
        store_row_stream<NQ, G>(Y + row * ldy + c0, qok, acc);
    }
}

int env_int(const char *name, int dflt)
{
    const char *v = std::getenv(name);
    if (!v || !*v) return dflt;
    int x = std::atoi(v);
    return x > 0 ? x : dflt;
}

struct FastShape {
    int cpl, g;
    int64_t slices;
    bool full;
};

// Lane shape for natural-order kernels: 8 or 16 columns per lane (more rows
// per wave), a group never wider than 64 lanes.
bool fast_shape(const float *X, int64_t ldx, const float *Y, int64_t ldy, int64_t F, FastShape &sh)
{
    auto al = [](const void *p) { return ((uintptr_t)p % 16) == 0; };
    if (F % 4 || ldx % 4 || ldy % 4 || !al(X) || !al(Y)) return false;
    // measured: 8 columns per lane is best up to F = 128, 16 beyond
    int cpl = env_int("GS_FAST_CPL", F <= 128 ? 8 : 16);
    if (cpl != 4 && cpl != 8 && cpl != 16) cpl = 16;
    while (cpl > 4 && F < 4 * (int64_t)cpl) cpl /= 2;  // at least 4 lanes per group
    int64_t lanes = ceil_div(F, cpl);
    int g = lanes <= 4 ? 4 : lanes <= 8 ? 8 : lanes <= 16 ? 16 : lanes <= 32 ? 32 : 64;
    sh.cpl = cpl;
    sh.g = g;
    sh.slices = ceil_div(F, (int64_t)g * cpl);
    sh.full = F % ((int64_t)g * cpl) == 0;
    return true;
}

template <class Fn>
bool dispatch_fast(const FastShape &sh, Fn &&fn)
{
#define GS_C(C, GG)                                                                              \
    if (sh.cpl == C && sh.g == GG) {                                                             \
        if (sh.full)                                                                             \
            fn(std::integral_constant<int, C>{}, std::integral_constant<int, GG>{}, std::true_type{}); \
        else                                                                                     \
            fn(std::integral_constant<int, C>{}, std::integral_constant<int, GG>{}, std::false_type{}); \
        return true;                                                                             \
    }
    GS_C(16, 4) GS_C(16, 8) GS_C(16, 16) GS_C(16, 32) GS_C(16, 64)
    GS_C(8, 4) GS_C(8, 8) GS_C(8, 16) GS_C(8, 32) GS_C(8, 64)
    GS_C(4, 4) GS_C(4, 8) GS_C(4, 16) GS_C(4, 32) GS_C(4, 64)
#undef GS_C
    return false;
}

// Measured on the mesh and block workloads: 8 resident-workgroup multiples
// (about one row tile per workgroup) beat a tighter persistent grid.
unsigned persistent_grid(int64_t tiles, int64_t slices)
{
    const int64_t cap = (int64_t)resident_workgroups() * env_int("GS_WG_MULT", 8);
    int64_t g = std::min(tiles, std::max<int64_t>(1, cap / std::max<int64_t>(1, slices)));
    return (unsigned)std::max<int64_t>(1, g);
}

}  // namespace

bool spmm_ell_fast(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                   hipStream_t s)
{
    FastShape sh;
    if (!fast_shape(X, ldx, Y, ldy, F, sh)) return false;
    return dispatch_fast(sh, [&](auto c_t, auto g_t, auto f_t) {
        constexpr int CPL = decltype(c_t)::value, G = decltype(g_t)::value;
        constexpr bool FU = decltype(f_t)::value;
        int T = 0, h = 0;
        if (m.K <= kChainFold && pick_window(m, (int64_t)G * CPL * 4, T, h)) {
            const int64_t ntiles = ceil_div(m.R, T);
            const size_t lds = (size_t)(T + 2 * h) * G * CPL * 4;
            dim3 grid(persistent_grid(ntiles, sh.slices), (unsigned)sh.slices);
            k_ell_window<CPL, G, FU><<<grid, kBlock, lds, s>>>(m.R, m.C, m.K, m.ell_col.as<int32_t>(),
                                                              m.ell_val.as<float>(), X, ldx, Y, ldy, F, T, h,
                                                              ntiles);
            GS_HIP(hipGetLastError());
            return;
        }
        const int64_t tiles = ceil_div(m.R, kBlock / G);
        dim3 grid(persistent_grid(tiles, sh.slices), (unsigned)sh.slices);
        if (m.K > kChainFold)
            k_ell_fast<CPL, G, FU, true><<<grid, kBlock, 0, s>>>(m.R, m.K, m.ell_col.as<int32_t>(),
                                                                  m.ell_val.as<float>(), X, ldx, Y, ldy, F);
        else
            k_ell_fast<CPL, G, FU, false><<<grid, kBlock, 0, s>>>(m.R, m.K, m.ell_col.as<int32_t>(),
                                                                   m.ell_val.as<float>(), X, ldx, Y, ldy, F);
        GS_HIP(hipGetLastError());
    });
}

bool spmm_dia_fast(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                   hipStream_t s)
{
    FastShape sh;
    if (!fast_shape(X, ldx, Y, ldy, F, sh)) return false;
    return dispatch_fast(sh, [&](auto c_t, auto g_t, auto f_t) {
        constexpr int CPL = decltype(c_t)::value, G = decltype(g_t)::value;
        constexpr bool FU = decltype(f_t)::value;
        const int64_t tiles = ceil_div(m.R, kBlock / G);
        dim3 grid(persistent_grid(tiles, sh.slices), (unsigned)sh.slices);
        if (m.ND > kChainFold)
            k_dia_fast<CPL, G, FU, true><<<grid, kBlock, 0, s>>>(m.R, m.C, m.ND, m.offsets.as<int32_t>(),
                                                                  m.dia.as<float>(), X, ldx, Y, ldy, F);
        else
            k_dia_fast<CPL, G, FU, false><<<grid, kBlock, 0, s>>>(m.R, m.C, m.ND, m.offsets.as<int32_t>(),
                                                                   m.dia.as<float>(), X, ldx, Y, ldy, F);
        GS_HIP(hipGetLastError());
    });
}

}  // namespace gs
