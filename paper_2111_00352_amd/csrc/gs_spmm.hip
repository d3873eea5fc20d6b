// SpMM Y = A.X for each storage format (the aggregation of a GNN layer,
// Sec. 2.1; formats of Sec. 2.2).  fp32 in and out, fused multiply-add.
//
// Shared layout of every kernel: a "row group" of G lanes (G in {8,16,32,64},
// always inside one 64-wide wavefront) owns one output row slice of G*VEC
// columns, lane l holding columns l*VEC .. l*VEC+VEC-1 as one vector; X rows
// are gathered with one VEC-wide load per lane, so a group reads G*VEC*4
// contiguous bytes of an X row per nonzero (256 B at F = 64 up to 1 KiB at
// F = 256).  grid.y walks F in slices of G*VEC columns when F is wider.
// Index/value streams are read once and are loaded cooperatively by the
// group (one entry per lane) and broadcast with cross-lane shuffles.
//
// Every sequential fp32 chain is bounded (row chunks of at most 256 terms,
// four interleaved accumulators), which keeps the rounding error far below
// 1e-5 |A||X|; partial sums of split rows are combined in a fixed order, so
// results are deterministic.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <vector>

#include "gs_device.h"
#include "gs_gather.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kBlock = 256;  // threads per workgroup for every SpMM kernel

template <int VEC>
struct Acc {
    float v[VEC];
    __device__ __forceinline__ void zero()
    {
#pragma unroll
        for (int i = 0; i < VEC; i++) v[i] = 0.0f;
    }
    __device__ __forceinline__ void fma(float a, const Vec<VEC> &x)
    {
#pragma unroll
        for (int i = 0; i < VEC; i++) v[i] = __builtin_fmaf(a, x.v[i], v[i]);
    }
    __device__ __forceinline__ void add(const Acc &o)
    {
#pragma unroll
        for (int i = 0; i < VEC; i++) v[i] += o.v[i];
    }
    __device__ __forceinline__ Vec<VEC> vec() const
    {
        Vec<VEC> r;
#pragma unroll
        for (int i = 0; i < VEC; i++) r.v[i] = v[i];
        return r;
    }
};

// Accumulates sum_{k in [k0,k1)} val[k] * X[col[k], c0 .. c0+VEC) for one
// group.  Entries are fetched G at a time (one per lane) and broadcast;
// four independent accumulators keep four X-row loads in flight per lane.
template <int VEC, int G>
__device__ __forceinline__ Acc<VEC> gather_range(const int32_t *__restrict__ col,
                                                 const float *__restrict__ val, int64_t k0,
                                                 int64_t k1, const float *__restrict__ X,
                                                 int64_t ldx, int64_t c0, bool active, int lane)
{
    Acc<VEC> a0, a1, a2, a3;
    a0.zero();
    a1.zero();
    a2.zero();
    a3.zero();
    for (int64_t kb = k0; kb < k1; kb += G) {
        const int64_t k = kb + lane;
        int cj = 0;
        float vj = 0.0f;
        if (k < k1) {
            cj = ld_stream(col + k);
            vj = ld_stream(val + k);
        }
        const int n = (int)((k1 - kb) < G ? (k1 - kb) : G);
        int j = 0;
        for (; j + 4 <= n; j += 4) {
            const int c_0 = __shfl(cj, j, G), c_1 = __shfl(cj, j + 1, G);
            const int c_2 = __shfl(cj, j + 2, G), c_3 = __shfl(cj, j + 3, G);
            const float v_0 = __shfl(vj, j, G), v_1 = __shfl(vj, j + 1, G);
            const float v_2 = __shfl(vj, j + 2, G), v_3 = __shfl(vj, j + 3, G);
            if (active) {
                const Vec<VEC> x0 = ld_vec<VEC>(X + (int64_t)c_0 * ldx + c0);
                const Vec<VEC> x1 = ld_vec<VEC>(X + (int64_t)c_1 * ldx + c0);
                const Vec<VEC> x2 = ld_vec<VEC>(X + (int64_t)c_2 * ldx + c0);
                const Vec<VEC> x3 = ld_vec<VEC>(X + (int64_t)c_3 * ldx + c0);
                a0.fma(v_0, x0);
                a1.fma(v_1, x1);
                a2.fma(v_2, x2);
                a3.fma(v_3, x3);
            }
        }
        for (; j < n; j++) {
            const int c_0 = __shfl(cj, j, G);
            const float v_0 = __shfl(vj, j, G);
            if (active) a0.fma(v_0, ld_vec<VEC>(X + (int64_t)c_0 * ldx + c0));
        }
    }
    a0.add(a1);
    a2.add(a3);
    a0.add(a2);
    return a0;
}

// ---------------------------------------------------------------- CSR
// Generic path (any F and alignment): one group per work item {row, start,
// len, slot} of the CSR plan; slot >= 0 items are chunks of long rows whose
// partial sums go to work[slot * F + c].

template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_csr_items_generic(
    int64_t n_items, const int4 *__restrict__ items, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ X, int64_t ldx, float *__restrict__ Y,
    int64_t ldy, int64_t F, float *__restrict__ work)
{
    constexpr int GPB = kBlock / G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * VEC) + (int64_t)lane * VEC;
    const bool active = c0 < F;
    const int64_t it = (int64_t)blockIdx.x * GPB + g;
    if (it >= n_items) return;
    const int4 d = items[it];
    // rows of the group tier are summed kChainFold entries at a time
    Acc<VEC> acc;
    acc.zero();
    for (int64_t cs = d.y, e = (int64_t)d.y + d.z; cs < e; cs += kChainFold)
        acc.add(gather_range<VEC, G>(col, val, cs, cs + kChainFold < e ? cs + kChainFold : e, X, ldx, c0, active,
                                     lane));
    if (!active) return;
    if (d.w < 0)
        st_vec_stream<VEC>(Y + (int64_t)d.x * ldy + c0, acc.vec());
    else
        st_vec<VEC>(work + (int64_t)d.w * F + c0, acc.vec());
}

// One group per long row: sums its chunks' partials in chunk order.
template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_csr_combine(const int32_t *__restrict__ long_rows,
                                                        const int32_t *__restrict__ long_first,
                                                        int64_t n_long, const float *__restrict__ work,
                                                        float *__restrict__ Y, int64_t ldy, int64_t F)
{
    constexpr int GPB = kBlock / G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * VEC) + (int64_t)lane * VEC;
    const int64_t lr = (int64_t)blockIdx.x * GPB + g;
    if (lr >= n_long || c0 >= F) return;
    Acc<VEC> acc;
    acc.zero();
    for (int64_t ch = long_first[lr]; ch < long_first[lr + 1]; ch++) {
        const Vec<VEC> p = ld_vec<VEC>(work + ch * F + c0);
#pragma unroll
        for (int i = 0; i < VEC; i++) acc.v[i] += p.v[i];
    }
    st_vec_stream<VEC>(Y + (int64_t)long_rows[lr] * ldy + c0, acc.vec());
}

// ---------------------------------------------------------------- COO
// Segmented reduction over the (row, col)-sorted triplets.  The entries are
// cut into T ranges of about per entries, each boundary q*per moved forward
// to the first row start within S entries (a row of at most S entries is
// never cut; a longer one may be), so group q's range is [snap(q*per),
// snap((q+1)*per)) and all groups have the same work, within S entries,
// whatever the row lengths.  S = per / 3 (4 to 32) when most entries lie
// near the diagonal, where rows are short and alike; else 0, exact ranges.  T is one round of the lane groups resident on the chip, or,
// when most entries lie near the diagonal, as many rounds as give ranges of
// about 110 entries: the groups at work at any moment then cover one band
// of rows, which share their X rows in L2.
// Row boundaries inside a range are found with a ballot over "row differs
// from the previous entry"; a segment is written straight to Y unless its
// row continues into a neighbouring range, in which case its partial goes to
// a carry slot: slot H (index 0) for the range's first segment when that row
// began in an earlier range, slot T (index 1) for the range's last segment
// when its row begins there and continues.  Inside a segment the running sum
// is folded every CH entries into a second sum (FOLD: only when a range can
// hold more than CH entries), so no fp32 chain is longer than CH plus the
// number of folds.  The boundaries, and for each range the split row it
// begins (its last row, continuing past it, or -1) with the number of later
// ranges the row runs into, depend only on the matrix and (T, per, S):
// they are computed once per handle and key.  k_coo_fixup then adds each
// split row's carries in range order.

// Range boundaries b[q] = the first row start in [q*per, q*per + S] (Z
// counts as one) or q*per itself, for q in [0, T] (b[0] = 0, b[T] = Z); then
// the split row each range begins: its last row when that row continues
// past the range and did not begin before it, else -1.
__global__ __launch_bounds__(kBlock) void k_coo_bounds(const int32_t *__restrict__ row, int64_t Z, int64_t per,
                                                       int S, int64_t T, int32_t *__restrict__ bounds)
{
    for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q <= T; q += (int64_t)gridDim.x * kBlock) {
        const int64_t p = q * per;
        int64_t b = p <= 0 ? 0 : p >= Z ? Z : -1;
        if (b < 0) {
            const int64_t lim = p + S < Z ? p + S : Z;
            b = p;
            for (int64_t k = p; k <= lim; k++)
                if (k == Z || row[k] != row[k - 1]) {
                    b = k;
                    break;
                }
        }
        bounds[q] = (int32_t)b;
    }
}

__global__ __launch_bounds__(kBlock) void k_coo_split_rows(const int32_t *__restrict__ row, int64_t Z, int64_t T,
                                                           const int32_t *__restrict__ bounds,
                                                           int4 *__restrict__ split, int32_t *__restrict__ flag)
{
    for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < T; q += (int64_t)gridDim.x * kBlock) {
        const int64_t k0 = bounds[q], k1 = bounds[q + 1];
        int4 d = make_int4((int)q, -1, 0, 0);
        if (k0 < k1 && k1 < Z && row[k1] == row[k1 - 1] && !(k0 > 0 && row[k0 - 1] == row[k1 - 1])) {
            // row r continues into ranges q+1 .. q+n: those whose first entry
            // is r (a prefix of the later ranges, found by bisection)
            const int32_t r = row[k1 - 1];
            int64_t lo = q + 1, hi = T;  // ranges q+1 .. lo-1 open with r; hi and later do not
            while (lo < hi) {
                const int64_t mid = (lo + hi) >> 1;
                const int64_t b = bounds[mid];
                if (b < Z && row[b] == r)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            d = make_int4((int)q, r, (int)(lo - q - 1), 0);
        }
        split[q] = d;
        flag[q] = d.y >= 0;
    }
}

// The ranges that begin a split row, in range order: split[q] for the q
// with flag (exclusive prefix pos).
__global__ __launch_bounds__(kBlock) void k_coo_split_list(const int4 *__restrict__ split, int64_t T,
                                                           const int32_t *__restrict__ pos,
                                                           int4 *__restrict__ list)
{
    for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < T; q += (int64_t)gridDim.x * kBlock)
        if (pos[q + 1] > pos[q]) list[pos[q]] = split[q];
}

template <int VEC>
__device__ __forceinline__ void coo_flush(const Acc<VEC> &acc, const Acc<VEC> &tot, bool folded, int64_t row,
                                          bool first_seg, bool last_seg, bool head_cont, bool tail_cont,
                                          int64_t q, float *__restrict__ Y, int64_t ldy,
                                          float *__restrict__ work, int64_t F, int64_t c0, bool active)
{
    if (!active) return;
    Acc<VEC> v = acc;
    if (folded) {
        v = tot;
        v.add(acc);
    }
    if (first_seg && head_cont)
        st_vec<VEC>(work + (q * 2 + 0) * F + c0, v.vec());
    else if (last_seg && tail_cont)
        st_vec<VEC>(work + (q * 2 + 1) * F + c0, v.vec());
    else
        st_vec_stream<VEC>(Y + row * ldy + c0, v.vec());
}

template <int VEC, int G, bool FOLD>
__global__ __launch_bounds__(kBlock) void k_coo_main(int64_t Z, const int32_t *__restrict__ row,
                                                     const int32_t *__restrict__ col,
                                                     const float *__restrict__ val,
                                                     const float *__restrict__ X, int64_t ldx,
                                                     float *__restrict__ Y, int64_t ldy, int64_t F,
                                                     const int32_t *__restrict__ bounds, int64_t per,
                                                     int64_t T, float *__restrict__ work)
{
    constexpr int GPB = kBlock / G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * VEC) + (int64_t)lane * VEC;
    const bool active = c0 < F;
    const int64_t q = xcd_tile(blockIdx.x, gridDim.x) * GPB + g;
    if (q >= T) return;
    const int gbase = (threadIdx.x % kWave) / G * G;  // first lane of this group in the wave
    int64_t k0, k1;
    if (bounds) {
        k0 = bounds[q];
        k1 = bounds[q + 1];
    } else {  // exact ranges
        k0 = q * per < Z ? q * per : Z;
        k1 = k0 + per < Z ? k0 + per : Z;
    }
    if (k0 >= k1) return;
    const bool head_cont = k0 > 0 && row[k0 - 1] == row[k0];
    const bool tail_cont = k1 < Z && row[k1] == row[k1 - 1];

    Acc<VEC> acc, tot;
    acc.zero();
    tot.zero();
    bool folded = false;
    int nin = 0;  // entries in acc since the segment began or acc was last folded
    int64_t cur = row[k0];
    bool first_seg = true;
    for (int64_t kb = k0; kb < k1; kb += G) {
        const int64_t k = kb + lane;
        int rj = -1, cj = 0;
        float vj = 0.0f;
        if (k < k1) {
            rj = ld_stream(row + k);
            cj = ld_stream(col + k);
            vj = ld_stream(val + k);
        }
        // bit j set: entry kb+j starts a new row relative to entry kb+j-1
        const int rprev = __shfl(rj, lane == 0 ? 0 : lane - 1, G);
        const bool starts = (k < k1) && lane > 0 && rj != rprev;
        const unsigned long long heads =
            (__ballot(starts) >> gbase) & (G == 64 ? ~0ull : ((1ull << G) - 1));
        const int n = (int)((k1 - kb) < G ? (k1 - kb) : G);
        // X rows of UB entries are requested before any of them is consumed;
        // entries past n gather row 0 of X (a valid row) and are skipped.
        constexpr int UB = 8;
        for (int j0 = 0; j0 < n; j0 += UB) {
            Vec<VEC> xs[UB];
            float vs[UB];
            int rs[UB];
#pragma unroll
            for (int u = 0; u < UB; u++) {
                const int j = j0 + u;
                const int c_u = __shfl(cj, j, G);
                vs[u] = __shfl(vj, j, G);
                rs[u] = __shfl(rj, j, G);
                if (active) xs[u] = ld_vec<VEC>(X + (int64_t)c_u * ldx + c0);
            }
#pragma unroll
            for (int u = 0; u < UB; u++) {
                const int j = j0 + u;
                if (j >= n) break;
                if ((j == 0 && rs[u] != cur) || ((heads >> j) & 1ull)) {
                    // the row changes before entry j: flush the finished segment
                    coo_flush<VEC>(acc, tot, folded, cur, first_seg, false, head_cont, tail_cont, q, Y, ldy,
                                   work, F, c0, active);
                    first_seg = false;
                    acc.zero();
                    tot.zero();
                    folded = false;
                    nin = 0;
                    cur = rs[u];
                }
                if (active) acc.fma(vs[u], xs[u]);
                if (FOLD && ++nin == kCooFold) {
                    tot.add(acc);
                    acc.zero();
                    folded = true;
                    nin = 0;
                }
            }
        }
    }
    coo_flush<VEC>(acc, tot, folded, cur, first_seg, true, head_cont, tail_cont, q, Y, ldy, work, F, c0,
                   active);
}

// The same ranges, segments and carry slots in the lane layout of the
// vectorised CSR kernels (F a multiple of 4, 16-byte aligned operands): lane
// l of a group holds NQ float4 at columns c0 + 4*G*q, so the per-entry
// shuffles and row-change tests serve 4*NQ columns of a lane instead of VEC,
// and the X rows of UB entries (8 float4 loads per lane) are requested
// before the first is consumed.
template <int NQ, int G>
__device__ __forceinline__ void coo_flush4(const float *acc, const float *tot, bool folded, int64_t row,
                                           bool first_seg, bool last_seg, bool head_cont, bool tail_cont,
                                           int64_t q, float *__restrict__ Y, int64_t ldy,
                                           float *__restrict__ work, int64_t F, int64_t c0, const bool *qok)
{
    float v[4 * NQ];
#pragma unroll
    for (int i = 0; i < 4 * NQ; i++) v[i] = folded ? tot[i] + acc[i] : acc[i];
    if (first_seg && head_cont)
        store_row<NQ, G>(work + (q * 2 + 0) * F + c0, qok, v);
    else if (last_seg && tail_cont)
        store_row<NQ, G>(work + (q * 2 + 1) * F + c0, qok, v);
    else
        store_row_stream<NQ, G>(Y + row * ldy + c0, qok, v);
}

template <int NQ, int G, bool FOLD>
__global__ __launch_bounds__(kBlock) void k_coo_main4(int64_t Z, const int32_t *__restrict__ row,
                                                      const int32_t *__restrict__ col,
                                                      const float *__restrict__ val,
                                                      const float *__restrict__ X, int64_t ldx,
                                                      float *__restrict__ Y, int64_t ldy, int64_t F,
                                                      const int32_t *__restrict__ bounds, int64_t per,
                                                      int64_t T, float *__restrict__ work)
{
    constexpr int GPB = kBlock / G;
    constexpr int UB = NQ >= 4 ? 2 : NQ == 2 ? 4 : 8;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (4 * G * NQ) + (int64_t)lane * 4;
    bool qok[NQ];
#pragma unroll
    for (int i = 0; i < NQ; i++) qok[i] = c0 + 4 * G * i < F;
    const int64_t q = xcd_tile(blockIdx.x, gridDim.x) * GPB + g;
    if (q >= T) return;
    const int gbase = (threadIdx.x % kWave) / G * G;
    int64_t k0, k1;
    if (bounds) {
        k0 = bounds[q];
        k1 = bounds[q + 1];
    } else {
        k0 = q * per < Z ? q * per : Z;
        k1 = k0 + per < Z ? k0 + per : Z;
    }
    if (k0 >= k1) return;
    const bool head_cont = k0 > 0 && row[k0 - 1] == row[k0];
    const bool tail_cont = k1 < Z && row[k1] == row[k1 - 1];

    float acc[4 * NQ], tot[4 * NQ];
#pragma unroll
    for (int i = 0; i < 4 * NQ; i++) acc[i] = tot[i] = 0.0f;
    bool folded = false;
    int nin = 0;
    int64_t cur = row[k0];
    bool first_seg = true;
    for (int64_t kb = k0; kb < k1; kb += G) {
        const int64_t k = kb + lane;
        int rj = -1, cj = 0;
        float vj = 0.0f;
        if (k < k1) {
            rj = ld_stream(row + k);
            cj = ld_stream(col + k);
            vj = ld_stream(val + k);
        }
        const int rprev = __shfl(rj, lane == 0 ? 0 : lane - 1, G);
        const bool starts = (k < k1) && lane > 0 && rj != rprev;
        const unsigned long long heads =
            (__ballot(starts) >> gbase) & (G == 64 ? ~0ull : ((1ull << G) - 1));
        const int n = (int)((k1 - kb) < G ? (k1 - kb) : G);
        // entries past n gather row 0 of X (cj = 0: a valid row) and are skipped
        for (int j0 = 0; j0 < n; j0 += UB) {
            float4 xs[UB][NQ];
            float vs[UB];
            int rs[UB];
#pragma unroll
            for (int u = 0; u < UB; u++) {
                const int c_u = __shfl(cj, j0 + u, G);
                vs[u] = __shfl(vj, j0 + u, G);
                rs[u] = __shfl(rj, j0 + u, G);
                const float *xp = X + (int64_t)c_u * ldx + c0;
#pragma unroll
                for (int i = 0; i < NQ; i++)
                    xs[u][i] = qok[i] ? load_x4(xp + 4 * G * i) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int u = 0; u < UB; u++) {
                const int j = j0 + u;
                if (j >= n) break;
                if ((j == 0 && rs[u] != cur) || ((heads >> j) & 1ull)) {
                    coo_flush4<NQ, G>(acc, tot, folded, cur, first_seg, false, head_cont, tail_cont, q, Y, ldy,
                                      work, F, c0, qok);
                    first_seg = false;
#pragma unroll
                    for (int i = 0; i < 4 * NQ; i++) acc[i] = tot[i] = 0.0f;
                    folded = false;
                    nin = 0;
                    cur = rs[u];
                }
#pragma unroll
                for (int i = 0; i < NQ; i++) {
                    acc[4 * i + 0] = __builtin_fmaf(vs[u], xs[u][i].x, acc[4 * i + 0]);
                    acc[4 * i + 1] = __builtin_fmaf(vs[u], xs[u][i].y, acc[4 * i + 1]);
                    acc[4 * i + 2] = __builtin_fmaf(vs[u], xs[u][i].z, acc[4 * i + 2]);
                    acc[4 * i + 3] = __builtin_fmaf(vs[u], xs[u][i].w, acc[4 * i + 3]);
                }
                if (FOLD && ++nin == kCooFold) {
#pragma unroll
                    for (int i = 0; i < 4 * NQ; i++) {
                        tot[i] += acc[i];
                        acc[i] = 0.0f;
                    }
                    folded = true;
                    nin = 0;
                }
            }
        }
    }
    coo_flush4<NQ, G>(acc, tot, folded, cur, first_seg, true, head_cont, tail_cont, q, Y, ldy, work, F, c0, qok);
}

// Groups [0, n_split): split row e = {range q, row r, n, 0}: range q begins
// row r, which continues into the next n ranges; the group adds slot T of q
// and then slot H of q+1 .. q+n in range order, sixteen loads in flight,
// and writes Y.  The groups after those zero the empty rows.
template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_coo_fixup(int64_t n_split, const int4 *__restrict__ split,
                                                      const float *__restrict__ work,
                                                      const int32_t *__restrict__ empty_rows,
                                                      int64_t n_empty, float *__restrict__ Y,
                                                      int64_t ldy, int64_t F)
{
    constexpr int GPB = kBlock / G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * VEC) + (int64_t)lane * VEC;
    const int64_t e = (int64_t)blockIdx.x * GPB + g;
    if (c0 >= F) return;
    if (e < n_split) {
        const int4 d4 = split[e];
        const int64_t q = d4.x;
        const int2 d = make_int2(d4.y, d4.z);
        Acc<VEC> acc;
        const Vec<VEC> t = ld_vec<VEC>(work + (q * 2 + 1) * F + c0);
#pragma unroll
        for (int i = 0; i < VEC; i++) acc.v[i] = t.v[i];
        // each batch of B carries is summed as a tree (zeros past the last)
        // before it joins the running sum: a row cut across n ranges adds
        // log2(B) + n / B terms in sequence, not n
        constexpr int B = 16;
        for (int64_t p0 = 1; p0 <= d.y; p0 += B) {
            Vec<VEC> h[B];
#pragma unroll
            for (int u = 0; u < B; u++) {
                if (p0 + u <= d.y) {
                    h[u] = ld_vec<VEC>(work + ((q + p0 + u) * 2 + 0) * F + c0);
                } else {
#pragma unroll
                    for (int i = 0; i < VEC; i++) h[u].v[i] = 0.0f;
                }
            }
#pragma unroll
            for (int w = 1; w < B; w <<= 1)
#pragma unroll
                for (int u = 0; u < B; u += 2 * w)
#pragma unroll
                    for (int i = 0; i < VEC; i++) h[u].v[i] += h[u + w].v[i];
#pragma unroll
            for (int i = 0; i < VEC; i++) acc.v[i] += h[0].v[i];
        }
        st_vec_stream<VEC>(Y + (int64_t)d.x * ldy + c0, acc.vec());
    } else {
        const int64_t k = e - n_split;
        if (k >= n_empty) return;
        Vec<VEC> z;
#pragma unroll
        for (int i = 0; i < VEC; i++) z.v[i] = 0.0f;
        st_vec_stream<VEC>(Y + (int64_t)empty_rows[k] * ldy + c0, z);
    }
}

// ---------------------------------------------------------------- CSC
// Column j of A scatters a_ij * X[j,:] into row i of Y for each of its
// entries, so rows are summed by many workgroups at once.  The products are
// exact in fp64 (24-bit mantissas), they are added with fp64 atomics into a
// workspace W (R x F doubles), and W is rounded to Y once: the fp64 sums
// carry no error that matters at fp32, whatever their order.  One wave per
// column, lanes over the F columns of X.

__global__ __launch_bounds__(kBlock) void k_fill_f64(double *__restrict__ w, int64_t n)
{
    for (int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x; k < n;
         k += (int64_t)gridDim.x * kBlock)
        w[k] = 0.0;
}

__global__ __launch_bounds__(kBlock) void k_csc_scatter(int64_t C, const int32_t *__restrict__ cp,
                                                        const int32_t *__restrict__ ri,
                                                        const float *__restrict__ val,
                                                        const float *__restrict__ X, int64_t ldx,
                                                        int64_t F, double *__restrict__ W)
{
    const int lane = threadIdx.x % kWave;
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t j = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / kWave; j < C; j += waves) {
        const int32_t k0 = cp[j], k1 = cp[j + 1];
        if (k0 == k1) continue;
        for (int64_t c0 = 0; c0 < F; c0 += 2 * kWave) {  // two X values per lane
            const int64_t ca = c0 + lane, cb = c0 + kWave + lane;
            const double xa = ca < F ? (double)X[j * ldx + ca] : 0.0;
            const double xb = cb < F ? (double)X[j * ldx + cb] : 0.0;
            // the column's entries 64 at a time: one row index and value per
            // lane, broadcast to the wave by shuffles
            for (int32_t kb = k0; kb < k1; kb += kWave) {
                const int n = k1 - kb < kWave ? k1 - kb : kWave;
                const int32_t rl = lane < n ? ri[kb + lane] : 0;
                const float vl = lane < n ? val[kb + lane] : 0.0f;
                for (int u = 0; u < n; u++) {
                    const int64_t r = __shfl(rl, u);
                    const double v = (double)__shfl(vl, u);
                    if (ca < F) unsafeAtomicAdd(&W[r * F + ca], v * xa);
                    if (cb < F) unsafeAtomicAdd(&W[r * F + cb], v * xb);
                }
            }
        }
    }
}

__global__ __launch_bounds__(kBlock) void k_round_f64(const double *__restrict__ W, int64_t R,
                                                      int64_t F, float *__restrict__ Y, int64_t ldy)
{
    for (int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x; k < R * F;
         k += (int64_t)gridDim.x * kBlock)
        Y[(k / F) * ldy + k % F] = (float)W[k];
}

// ---------------------------------------------------------------- ELL
// One group per row; slot (i,k) lives at k*R + i, so for a fixed k the
// groups of a block read consecutive addresses.  Padding (col = -1) ends
// the row (entries are packed to the front).

template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_ell(int64_t R, int64_t K, const int32_t *__restrict__ ec,
                                                const float *__restrict__ ev,
                                                const float *__restrict__ X, int64_t ldx,
                                                float *__restrict__ Y, int64_t ldy, int64_t F,
                                                int64_t n_tiles)
{
    constexpr int GPB = kBlock / G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * VEC) + (int64_t)lane * VEC;
    const bool active = c0 < F;
    const int64_t row = xcd_tile(blockIdx.x, n_tiles) * GPB + g;
    if (row >= R) return;
    const int gbase = (threadIdx.x % kWave) / G * G;
    Acc<VEC> a0, a1, tot;
    a0.zero();
    a1.zero();
    tot.zero();
    for (int64_t kb = 0; kb < K; kb += G) {
        if (kb > 0 && kb % kChainFold == 0) {  // fold the running chains every kChainFold slots
            tot.add(a0);
            tot.add(a1);
            a0.zero();
            a1.zero();
        }
        const int64_t k = kb + lane;
        int cj = -1;
        float vj = 0.0f;
        if (k < K) {
            cj = ld_stream(ec + k * R + row);
            vj = ld_stream(ev + k * R + row);
        }
        // entries are packed to the front: the stored ones form a prefix
        const unsigned long long live =
            (__ballot(cj >= 0) >> gbase) & (G == 64 ? ~0ull : ((1ull << G) - 1));
        const int n = __popcll(live);
        int j = 0;
        for (; j + 2 <= n; j += 2) {
            const int c_0 = __shfl(cj, j, G), c_1 = __shfl(cj, j + 1, G);
            const float v_0 = __shfl(vj, j, G), v_1 = __shfl(vj, j + 1, G);
            if (active) {
                const Vec<VEC> x0 = ld_vec<VEC>(X + (int64_t)c_0 * ldx + c0);
                const Vec<VEC> x1 = ld_vec<VEC>(X + (int64_t)c_1 * ldx + c0);
                a0.fma(v_0, x0);
                a1.fma(v_1, x1);
            }
        }
        if (j < n) {
            const int c_0 = __shfl(cj, j, G);
            const float v_0 = __shfl(vj, j, G);
            if (active) a0.fma(v_0, ld_vec<VEC>(X + (int64_t)c_0 * ldx + c0));
        }
        if (n < G) break;
    }
    tot.add(a0);
    tot.add(a1);
    if (active) st_vec_stream<VEC>(Y + row * ldy + c0, tot.vec());
}

// ---------------------------------------------------------------- DIA
// One group per row; diagonal d contributes data[d*R+i] * X[i + off_d].
// Padding slots hold +0 and are skipped, as are columns outside [0, C).

template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_dia(int64_t R, int64_t C, int64_t ND,
                                                const int32_t *__restrict__ offsets,
                                                const float *__restrict__ data,
                                                const float *__restrict__ X, int64_t ldx,
                                                float *__restrict__ Y, int64_t ldy, int64_t F,
                                                int64_t n_tiles)
{
    constexpr int GPB = kBlock / G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * VEC) + (int64_t)lane * VEC;
    const bool active = c0 < F;
    const int64_t row = xcd_tile(blockIdx.x, n_tiles) * GPB + g;
    if (row >= R) return;
    Acc<VEC> a0, a1, tot;
    a0.zero();
    a1.zero();
    tot.zero();
    int64_t d = 0;
    for (; d + 2 <= ND; d += 2) {
        if (d > 0 && d % kChainFold == 0) {  // fold the running chains every kChainFold diagonals
            tot.add(a0);
            tot.add(a1);
            a0.zero();
            a1.zero();
        }
        const int64_t j0 = row + offsets[d], j1 = row + offsets[d + 1];
        const float v0 = ld_stream(data + d * R + row);
        const float v1 = ld_stream(data + (d + 1) * R + row);
        if (active) {
            if (v0 != 0.0f && j0 >= 0 && j0 < C) a0.fma(v0, ld_vec<VEC>(X + j0 * ldx + c0));
            if (v1 != 0.0f && j1 >= 0 && j1 < C) a1.fma(v1, ld_vec<VEC>(X + j1 * ldx + c0));
        }
    }
    if (d < ND) {
        const int64_t j0 = row + offsets[d];
        const float v0 = ld_stream(data + d * R + row);
        if (active && v0 != 0.0f && j0 >= 0 && j0 < C) a0.fma(v0, ld_vec<VEC>(X + j0 * ldx + c0));
    }
    tot.add(a0);
    tot.add(a1);
    if (active) st_vec_stream<VEC>(Y + row * ldy + c0, tot.vec());
}

// ---------------------------------------------------------------- BSR
// One workgroup per block row.  Lanes split F as everywhere else; the
// kBlock/G row groups split the b rows of the block row (each thread owns
// up to RPT rows).  Each b x b block is staged in LDS; only the block
// columns with a nonzero (bit set in the block's column mask) gather their
// X row, so a sparse block costs its b*b values plus its touched X rows.

template <int VEC, int G, int RPT>
__global__ __launch_bounds__(kBlock) void k_bsr(int64_t R, int64_t C, int b, int64_t nbr,
                                                const int32_t *__restrict__ bptr,
                                                const int32_t *__restrict__ bcol,
                                                const float *__restrict__ bval,
                                                const uint64_t *__restrict__ bmask,
                                                const float *__restrict__ X, int64_t ldx,
                                                float *__restrict__ Y, int64_t ldy, int64_t F)
{
    constexpr int RG = kBlock / G;  // row groups
    __shared__ float blk_lds[64 * 64];
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * VEC) + (int64_t)lane * VEC;
    const bool active = c0 < F;
    const int64_t br = xcd_tile(blockIdx.x, nbr);
    const int bb = b * b;
    Acc<VEC> acc[RPT], tot[RPT];
#pragma unroll
    for (int r = 0; r < RPT; r++) {
        acc[r].zero();
        tot[r].zero();
    }
    const int64_t fold = kChainFold / b > 0 ? kChainFold / b : 1;  // blocks per running chain
    for (int64_t blk = bptr[br]; blk < bptr[br + 1]; blk++) {
        if (blk > bptr[br] && (blk - bptr[br]) % fold == 0) {
#pragma unroll
            for (int r = 0; r < RPT; r++) {
                tot[r].add(acc[r]);
                acc[r].zero();
            }
        }
        __syncthreads();
        for (int t = threadIdx.x; t < bb; t += kBlock) blk_lds[t] = ld_stream(bval + blk * bb + t);
        __syncthreads();
        uint64_t mask = bmask[blk];
        const int64_t xc = (int64_t)bcol[blk] * b;
        while (mask) {
            const int j = __ffsll((unsigned long long)mask) - 1;
            mask &= mask - 1;
            if (!active) continue;
            const Vec<VEC> x = ld_vec<VEC>(X + (xc + j) * ldx + c0);
#pragma unroll
            for (int r = 0; r < RPT; r++) {
                const int rr = g + r * RG;
                if (rr < b) acc[r].fma(blk_lds[rr * b + j], x);
            }
        }
    }
    if (!active) return;
#pragma unroll
    for (int r = 0; r < RPT; r++) {
        tot[r].add(acc[r]);
        const int rr = g + r * RG;
        const int64_t row = br * b + rr;
        if (rr < b && row < R) st_vec_stream<VEC>(Y + row * ldy + c0, tot[r].vec());
    }
}

// ----------------------------------------------------------- dispatch

struct Shape {
    int vec;
    int g;
    int64_t fslices;  // grid.y
};

Shape pick_shape(const float *X, int64_t ldx, const float *Y, int64_t ldy, int64_t F)
{
    auto al = [](const void *p, int n) { return ((uintptr_t)p % n) == 0; };
    int vec = 1;
    if (F % 4 == 0 && ldx % 4 == 0 && ldy % 4 == 0 && al(X, 16) && al(Y, 16))
        vec = 4;
    else if (F % 2 == 0 && ldx % 2 == 0 && ldy % 2 == 0 && al(X, 8) && al(Y, 8))
        vec = 2;
    const int64_t lanes = ceil_div(F, vec);
    const int g = lanes <= 8 ? 8 : lanes <= 16 ? 16 : lanes <= 32 ? 32 : 64;
    return Shape{vec, g, ceil_div(F, (int64_t)g * vec)};
}

// Calls fn.template operator()<VEC, G>() for the runtime (vec, g).
template <class Fn>
void dispatch(const Shape &sh, Fn &&fn)
{
#define GS_CASE(V, GG) \
    if (sh.vec == V && sh.g == GG) return fn.template operator()<V, GG>();
    GS_CASE(4, 8) GS_CASE(4, 16) GS_CASE(4, 32) GS_CASE(4, 64)
    GS_CASE(2, 8) GS_CASE(2, 16) GS_CASE(2, 32) GS_CASE(2, 64)
    GS_CASE(1, 8) GS_CASE(1, 16) GS_CASE(1, 32) GS_CASE(1, 64)
#undef GS_CASE
    fail(GS_ERR_UNSUPPORTED, "no kernel for vec=%d g=%d", sh.vec, sh.g);
}

unsigned u32_grid(int64_t n)
{
    if (n > 0x7fffffffll) fail(GS_ERR_UNSUPPORTED, "grid of %lld workgroups is too large", (long long)n);
    return (unsigned)(n < 1 ? 1 : n);
}

}  // namespace

// --------------------------------------------------------------- plans

// The COO plan lists the empty rows, which the SpMM must zero (the kernel
// writes only rows that hold entries), and counts the entries near the
// diagonal, which sets the number of rounds of ranges per SpMM.

namespace {

constexpr int kPB = 256;

inline unsigned plan_blocks(int64_t n)
{
    int64_t g = ceil_div(n, (int64_t)kPB);
    return (unsigned)(g < 1 ? 1 : g > 8192 ? 8192 : g);
}

__global__ __launch_bounds__(kPB) void k_empty_flags(const int32_t *__restrict__ rp, int64_t R,
                                                     int32_t *__restrict__ is_empty)
{
    for (int64_t i = (int64_t)blockIdx.x * kPB + threadIdx.x; i < R; i += (int64_t)gridDim.x * kPB)
        is_empty[i] = rp[i + 1] == rp[i];
}

__global__ __launch_bounds__(kPB) void k_empty_list(int64_t R, const int32_t *__restrict__ off,
                                                    int32_t *__restrict__ empty)
{
    for (int64_t i = (int64_t)blockIdx.x * kPB + threadIdx.x; i < R; i += (int64_t)gridDim.x * kPB)
        if (off[i + 1] > off[i]) empty[off[i]] = (int32_t)i;
}

// Entries with |col - row| < kCooNear, one partial per workgroup.
constexpr int64_t kCooNear = 4096;
__global__ __launch_bounds__(kPB) void k_coo_near(const int32_t *__restrict__ row, const int32_t *__restrict__ col,
                                                  int64_t Z, unsigned long long *__restrict__ part)
{
    __shared__ unsigned long long t64[kPB / kWave];
    unsigned long long n = 0;
    for (int64_t k = (int64_t)blockIdx.x * kPB + threadIdx.x; k < Z; k += (int64_t)gridDim.x * kPB) {
        const int64_t d = (int64_t)col[k] - row[k];
        n += d > -kCooNear && d < kCooNear;
    }
    n = block_sum_u64<kPB>(n, t64);
    if (threadIdx.x == 0) part[blockIdx.x] = n;
}

}  // namespace

void plan_coo(gs_matrix_ &m, const int32_t *row_ptr, hipStream_t s)
{
    const int64_t R = m.R, Z = m.Z;
    DevBuf emp, near;
    emp.alloc((size_t)(R + 1) * 4, s);
    near.alloc(sizeof(unsigned long long) * 2049, s);
    unsigned long long *d_near = near.as<unsigned long long>() + 2048;
    GS_HIP(hipMemsetAsync(d_near, 0, sizeof(unsigned long long), s));
    if (R > 0) {
        k_empty_flags<<<plan_blocks(R), kPB, 0, s>>>(row_ptr, R, emp.as<int32_t>());
        GS_HIP(hipGetLastError());
    }
    exclusive_scan_i32(emp.as<int32_t>(), emp.as<int32_t>(), R, true, s);
    if (Z > 0) {
        const unsigned G = (unsigned)std::min<int64_t>(2048, ceil_div(Z, (int64_t)kPB * 8));
        k_coo_near<<<G, kPB, 0, s>>>(m.row.as<int32_t>(), m.col.as<int32_t>(), Z, near.as<unsigned long long>());
        GS_HIP(hipGetLastError());
        add_partials_u64(near.as<unsigned long long>(), G, d_near, s);
    }
    int32_t n_empty = 0;
    unsigned long long n_near = 0;
    GS_HIP(hipMemcpyAsync(&n_empty, emp.as<int32_t>() + R, 4, hipMemcpyDeviceToHost, s));
    GS_HIP(hipMemcpyAsync(&n_near, d_near, sizeof n_near, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));
    m.coo_local = (int64_t)n_near;
    m.n_empty_rows = n_empty;
    m.empty_rows.alloc((size_t)n_empty * 4, s);
    if (n_empty) {
        k_empty_list<<<plan_blocks(R), kPB, 0, s>>>(R, emp.as<int32_t>(), m.empty_rows.as<int32_t>());
        GS_HIP(hipGetLastError());
    }
}

// --------------------------------------------------------------- launchers

void spmm_csr(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s, const WorkArea *fixed)
{
    if (!m.csr_planned) {
        if (fixed) fail(GS_ERR_UNSUPPORTED, "CSR handle without a work plan (it is built with the handle)");
        plan_csr(m, s);
    }
    if (spmm_csr_vec4(m, X, ldx, Y, ldy, F, s, fixed)) return;
    const Shape sh = pick_shape(X, ldx, Y, ldy, F);
    float *work = m.n_long_chunks ? (float *)work_for(m, fixed, (size_t)m.n_long_chunks * F * 4, s) : nullptr;
    dispatch(sh, [&]<int VEC, int G>() {
        constexpr int GPB = kBlock / G;
        if (m.n_items) {
            dim3 grid(u32_grid(ceil_div(m.n_items, GPB)), (unsigned)sh.fslices);
            k_csr_items_generic<VEC, G><<<grid, kBlock, 0, s>>>(
                m.n_items, m.csr_items.as<int4>(), m.col.as<int32_t>(), m.val.as<float>(), X, ldx, Y,
                ldy, F, work);
            GS_HIP(hipGetLastError());
        }
        if (m.n_long_rows) {
            dim3 g2(u32_grid(ceil_div(m.n_long_rows, GPB)), (unsigned)sh.fslices);
            k_csr_combine<VEC, G><<<g2, kBlock, 0, s>>>(m.long_rows.as<int32_t>(),
                                                        m.long_first.as<int32_t>(), m.n_long_rows,
                                                        work, Y, ldy, F);
            GS_HIP(hipGetLastError());
        }
    });
}

namespace {

using CooMainFn = void (*)(int64_t, const int32_t *, const int32_t *, const float *, const float *, int64_t,
                           float *, int64_t, int64_t, const int32_t *, int64_t, int64_t, float *);

// The main COO pass for one lane shape: its plain and folding variants, lane
// groups per workgroup and column slices of F.
struct CooMain {
    CooMainFn plain = nullptr, fold = nullptr;
    int gpb = 0;
    int64_t fslices = 0;
};

// float4 per lane of the vectorised pass: GS_COO_CPL (columns per lane: 4, 8
// or 16) where set.  Otherwise 8 columns per lane from F = 64 on while X fits
// in the 256 MiB memory-side cache; an X that does not is gathered from HBM,
// where 4 columns per lane (one wider load per X row) measured faster.
int coo_nq(int64_t C, int64_t F)
{
    if (const char *e = std::getenv("GS_COO_CPL")) {
        const int c = std::atoi(e);
        if (c == 4 || c == 8 || c == 16) return c / 4;
    }
    return F >= 64 && C * F * 4 <= (256ll << 20) ? 2 : 1;
}

template <int NQ, int G>
CooMain coo_main4()
{
    CooMain c;
    c.plain = k_coo_main4<NQ, G, false>;
    c.fold = k_coo_main4<NQ, G, true>;
    c.gpb = kBlock / G;
    return c;
}

CooMain pick_coo_main(const Shape &sh, int64_t C, int64_t F)
{
    CooMain c;
    const int nq = sh.vec == 4 ? coo_nq(C, F) : 1;
    if (nq > 1) {
        const int64_t lanes = ceil_div(F, (int64_t)4 * nq);
        const int g = lanes <= 8 ? 8 : lanes <= 16 ? 16 : lanes <= 32 ? 32 : 64;
#define GS_C4(N, GG) \
    if (nq == N && g == GG) c = coo_main4<N, GG>();
        GS_C4(2, 8) GS_C4(2, 16) GS_C4(2, 32) GS_C4(2, 64)
        GS_C4(4, 8) GS_C4(4, 16) GS_C4(4, 32) GS_C4(4, 64)
#undef GS_C4
        c.fslices = ceil_div(F, (int64_t)4 * g * nq);
        return c;
    }
    dispatch(sh, [&]<int VEC, int G>() {
        c.plain = k_coo_main<VEC, G, false>;
        c.fold = k_coo_main<VEC, G, true>;
        c.gpb = kBlock / G;
        c.fslices = sh.fslices;
    });
    return c;
}

// Resident workgroups per CU of a main-pass kernel.
int coo_occupancy(CooMainFn fn)
{
    static std::mutex mu;
    static std::map<CooMainFn, int> cache;
    std::lock_guard<std::mutex> lock(mu);
    auto it = cache.find(fn);
    if (it != cache.end()) return it->second;
    int n = 0;
    GS_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kBlock, 0));
    return cache[fn] = n > 0 ? n : 1;
}

}  // namespace

void spmm_coo(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s, const WorkArea *fixed)
{
    // the range tables are built (and allocated) per launch shape on first use
    if (fixed) fail(GS_ERR_UNSUPPORTED, "COO handles are not supported without allocation");
    const Shape sh = pick_shape(X, ldx, Y, ldy, F);
    const CooMain cm = pick_coo_main(sh, m.C, F);  // main pass; the fixup keeps the generic shape
    const int64_t Z = m.Z;
    dispatch(sh, [&]<int VEC, int G>() {
        constexpr int GPB = kBlock / G;
        int64_t T = 0, per = 0;
        int S = 0;
        const int32_t *bounds = nullptr;
        const int4 *split_list = nullptr;
        int64_t n_split = 0;
        if (Z > 0) {
            const bool local = 2 * m.coo_local >= Z;
            const char *force_T = std::getenv("GS_COO_RANGES");  // tests
            // ranges of one round of the resident lane groups (shared by the
            // F slices); as many rounds as give ranges of about kCooBandRange
            // entries when most entries lie near the diagonal.  Row-aligned
            // boundaries pay where rows are short and alike (near-diagonal
            // matrices); on random graphs the cut rows are long anyway, and
            // exact ranges keep the single round balanced.
            auto split = [&](int occ) {
                const int64_t round = std::max<int64_t>(1, (int64_t)occ * compute_units() * cm.gpb / cm.fslices);
                const int64_t rounds = local ? std::max<int64_t>(1, Z / (round * kCooBandRange)) : 1;
                T = std::min<int64_t>(rounds * round, ceil_div(Z, (int64_t)kCooMinRange));
                if (force_T && *force_T) T = std::max<int64_t>(1, std::atoll(force_T));
                per = ceil_div(Z, T);
                T = ceil_div(Z, per);  // no range past the last entry
                // (at most kCooFold - per where that leaves 4 or more: then no
                // range exceeds kCooFold entries and the launch needs no folds)
                S = 0;
                if (local) {
                    int64_t w = std::min<int64_t>(kCooSnap, per / 3);
                    if (kCooFold - per >= 4) w = std::min<int64_t>(w, kCooFold - per);
                    S = (int)std::max<int64_t>(4, w);
                }
                if (const char *e = std::getenv("GS_COO_SNAP"); e && *e)  // tests and tuning
                    S = (int)std::clamp<int64_t>(std::atoll(e), 0, kCooSnap);
            };
            split(coo_occupancy(cm.fold));
            if (per + S <= kCooFold) split(coo_occupancy(cm.plain));  // the launch will not fold: its own occupancy
            auto key = std::make_tuple(T, per, S);
            auto it = m.coo_ranges.find(key);
            if (it == m.coo_ranges.end()) {  // first call with this split: boundaries and split rows
                gs_matrix_::CooRanges cr;
                cr.bounds.alloc((size_t)(T + 1) * 4, s);
                DevBuf all, pos;
                all.alloc((size_t)T * sizeof(int4), s);
                pos.alloc((size_t)(T + 1) * 4, s);
                const unsigned gb = (unsigned)std::min<int64_t>(4096, ceil_div(T + 1, (int64_t)kBlock));
                k_coo_bounds<<<gb, kBlock, 0, s>>>(m.row.as<int32_t>(), Z, per, S, T, cr.bounds.as<int32_t>());
                GS_HIP(hipGetLastError());
                k_coo_split_rows<<<gb, kBlock, 0, s>>>(m.row.as<int32_t>(), Z, T, cr.bounds.as<int32_t>(),
                                                       all.as<int4>(), pos.as<int32_t>());
                GS_HIP(hipGetLastError());
                exclusive_scan_i32(pos.as<int32_t>(), pos.as<int32_t>(), T, true, s);
                int32_t ns = 0;
                GS_HIP(hipMemcpyAsync(&ns, pos.as<int32_t>() + T, 4, hipMemcpyDeviceToHost, s));
                GS_HIP(hipStreamSynchronize(s));
                cr.n_split = ns;
                cr.split.alloc((size_t)ns * sizeof(int4), s);
                if (ns) {
                    k_coo_split_list<<<gb, kBlock, 0, s>>>(all.as<int4>(), T, pos.as<int32_t>(), cr.split.as<int4>());
                    GS_HIP(hipGetLastError());
                }
                it = m.coo_ranges.emplace(key, std::move(cr)).first;
            }
            bounds = S ? it->second.bounds.as<int32_t>() : nullptr;  // exact ranges: q * per
            split_list = it->second.split.as<int4>();
            n_split = it->second.n_split;
            if (T > 1) ensure_work(m, (size_t)T * 2 * F * 4, s);  // two carry slots of F floats per range
            dim3 grid(u32_grid(ceil_div(T, (int64_t)cm.gpb)), (unsigned)cm.fslices);
            const CooMainFn fn = per + S > kCooFold ? cm.fold : cm.plain;
            fn<<<grid, kBlock, 0, s>>>(Z, m.row.as<int32_t>(), m.col.as<int32_t>(), m.val.as<float>(), X, ldx, Y,
                                       ldy, F, bounds, per, T, m.work.as<float>());
            GS_HIP(hipGetLastError());
        }
        const int64_t groups = n_split + m.n_empty_rows;
        if (groups) {
            dim3 g2(u32_grid(ceil_div(groups, GPB)), (unsigned)sh.fslices);
            k_coo_fixup<VEC, G><<<g2, kBlock, 0, s>>>(n_split, split_list, m.work.as<float>(),
                                                      m.empty_rows.as<int32_t>(), m.n_empty_rows, Y, ldy, F);
            GS_HIP(hipGetLastError());
        }
    });
}

void spmm_csc(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s, const WorkArea *fixed)
{
    const int64_t n = m.R * F;
    if (n == 0) return;
    double *W = (double *)work_for(m, fixed, (size_t)n * 8, s);
    auto grid = [](int64_t items) {
        int64_t g = ceil_div(items, (int64_t)kBlock);
        return (unsigned)(g < 1 ? 1 : g > 65536 ? 65536 : g);
    };
    k_fill_f64<<<grid(n), kBlock, 0, s>>>(W, n);
    GS_HIP(hipGetLastError());
    if (m.Z) {
        k_csc_scatter<<<grid(m.C * kWave), kBlock, 0, s>>>(m.C, m.row_ptr.as<int32_t>(), m.col.as<int32_t>(),
                                                             m.val.as<float>(), X, ldx, F, W);
        GS_HIP(hipGetLastError());
    }
    k_round_f64<<<grid(n), kBlock, 0, s>>>(W, m.R, F, Y, ldy);
    GS_HIP(hipGetLastError());
}

void spmm_ell(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s)
{
    if (spmm_ell_fast(m, X, ldx, Y, ldy, F, s)) return;
    const Shape sh = pick_shape(X, ldx, Y, ldy, F);
    dispatch(sh, [&]<int VEC, int G>() {
        constexpr int GPB = kBlock / G;
        const int64_t tiles = ceil_div(m.R, GPB);
        if (!tiles) return;
        dim3 grid(u32_grid(tiles), (unsigned)sh.fslices);
        k_ell<VEC, G><<<grid, kBlock, 0, s>>>(m.R, m.K, m.ell_col.as<int32_t>(), m.ell_val.as<float>(),
                                              X, ldx, Y, ldy, F, tiles);
        GS_HIP(hipGetLastError());
    });
}

void spmm_dia(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s)
{
    if (spmm_dia_fast(m, X, ldx, Y, ldy, F, s)) return;
    const Shape sh = pick_shape(X, ldx, Y, ldy, F);
    dispatch(sh, [&]<int VEC, int G>() {
        constexpr int GPB = kBlock / G;
        const int64_t tiles = ceil_div(m.R, GPB);
        if (!tiles) return;
        dim3 grid(u32_grid(tiles), (unsigned)sh.fslices);
        k_dia<VEC, G><<<grid, kBlock, 0, s>>>(m.R, m.C, m.ND, m.offsets.as<int32_t>(), m.dia.as<float>(),
                                              X, ldx, Y, ldy, F, tiles);
        GS_HIP(hipGetLastError());
    });
}

void spmm_bsr(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s)
{
    if (spmm_bsr16_mfma(m, X, ldx, Y, ldy, F, s)) return;
    const Shape sh = pick_shape(X, ldx, Y, ldy, F);
    const int64_t nbr = ceil_div(m.R, m.b);
    if (!nbr) return;
    dispatch(sh, [&]<int VEC, int G>() {
        constexpr int RG = kBlock / G;
        const int rpt = (int)ceil_div(m.b, RG);
        dim3 grid(u32_grid(nbr), (unsigned)sh.fslices);
        auto go = [&](auto rpt_tag) {
            constexpr int RPT = decltype(rpt_tag)::value;
            k_bsr<VEC, G, RPT><<<grid, kBlock, 0, s>>>(m.R, m.C, m.b, nbr, m.bptr.as<int32_t>(),
                                                       m.bcol.as<int32_t>(), m.bval.as<float>(),
                                                       m.bmask.as<uint64_t>(), X, ldx, Y, ldy, F);
        };
        if (rpt <= 1) go(std::integral_constant<int, 1>{});
        else if (rpt <= 2) go(std::integral_constant<int, 2>{});
        else if (rpt <= 4) go(std::integral_constant<int, 4>{});
        else if (rpt <= 8) go(std::integral_constant<int, 8>{});
        else go(std::integral_constant<int, 16>{});
        GS_HIP(hipGetLastError());
    });
}

}  // namespace gs
