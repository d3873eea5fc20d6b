// Matrix features of the format predictor (Sec. 4.4, Table 2), extracted on
// the device from the canonical CSR form.  The device produces integer
// aggregates only (row/column counts and their max, min, sum of squares and
// sum of adjacent absolute differences; the number of occupied diagonals;
// the number of occupied 16x16 blocks), combined with integer atomics, so
// the result is exact and deterministic.  The 19 doubles are then formed on
// the host from those integers in one fixed operation order.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdlib>

#include "gs_device.h"
#include "gs_host.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kTB = 256;

struct FeatAcc {
    unsigned long long s2r, s2c, bnr, bnc;
    int maxr, minr, maxc, minc;
};

inline unsigned elem_grid(int64_t n)
{
    int64_t g = ceil_div(n, kTB);
    if (g > 256 * 64) g = 256 * 64;
    if (g < 1) g = 1;
    return (unsigned)g;
}

__global__ __launch_bounds__(kTB) void k_col_hist(const int32_t *__restrict__ col, int64_t Z,
                                                  int32_t *__restrict__ cc)
{
    for (int64_t k = (int64_t)blockIdx.x * kTB + threadIdx.x; k < Z;
         k += (int64_t)gridDim.x * kTB)
        atomicAdd(&cc[col[k]], 1);
}

// Column counts without global atomics (large matrices): the column indices
// are first grouped by their high bits (buckets of 2^shift columns, so a
// bucket's counters fit in one workgroup's LDS), then every slice of a
// bucket is counted by one workgroup in LDS and written out whole, and the
// slices' counts are added per column.
constexpr int kBucketTile = kTB * 16;  // keys per tile of the bucketing passes
constexpr int kBucketPer = kBucketTile / kTB;

// hist[b * ntiles + t] = number of keys of tile t in bucket b.
__global__ __launch_bounds__(kTB) void k_bucket_hist(const uint32_t *__restrict__ keys, int64_t Z,
                                                     int shift, int nb, int64_t ntiles,
                                                     int32_t *__restrict__ hist)
{
    __shared__ int h[kTB];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kBucketTile;
    uint32_t v[kBucketPer];
#pragma unroll
    for (int i = 0; i < kBucketPer; i++) {  // all loads in flight before the counting
        const int64_t k = base + (int64_t)i * kTB + threadIdx.x;
        v[i] = k < Z ? keys[k] : ~0u;
    }
#pragma unroll
    for (int i = 0; i < kBucketPer; i++)
        if (v[i] != ~0u) atomicAdd(&h[v[i] >> shift], 1);
    __syncthreads();
    if (threadIdx.x < nb) hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

// Writes tile t's keys of bucket b from position off[b * ntiles + t] on.
// The tile is first grouped by bucket in LDS, so every bucket's keys leave
// as one contiguous run (order inside a bucket is free).
__global__ __launch_bounds__(kTB) void k_bucket_scatter(const uint32_t *__restrict__ keys, int64_t Z,
                                                        int shift, int nb, int64_t ntiles,
                                                        const int32_t *__restrict__ off,
                                                        uint32_t *__restrict__ out)
{
    __shared__ int cnt[kTB], lstart[kTB], gbase[kTB], tmp[kTB / kWave];
    __shared__ uint32_t stage[kBucketTile];
    cnt[threadIdx.x] = 0;
    if (threadIdx.x < nb) gbase[threadIdx.x] = off[(int64_t)threadIdx.x * ntiles + blockIdx.x];
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kBucketTile;
    uint32_t v[kBucketPer];
    int rank[kBucketPer];
#pragma unroll
    for (int i = 0; i < kBucketPer; i++) {
        const int64_t k = base + (int64_t)i * kTB + threadIdx.x;
        v[i] = k < Z ? keys[k] : ~0u;
    }
#pragma unroll
    for (int i = 0; i < kBucketPer; i++) rank[i] = v[i] != ~0u ? atomicAdd(&cnt[v[i] >> shift], 1) : 0;
    __syncthreads();
    lstart[threadIdx.x] = block_exclusive_scan<kTB>(cnt[threadIdx.x], tmp);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kBucketPer; i++)
        if (v[i] != ~0u) stage[lstart[v[i] >> shift] + rank[i]] = v[i];
    __syncthreads();
    const int n = (int)(Z - base < kBucketTile ? Z - base : kBucketTile);
    for (int j = threadIdx.x; j < n; j += kTB) {
        const uint32_t x = stage[j];
        const int bk = (int)(x >> shift);
        out[gbase[bk] + (j - lstart[bk])] = x;
    }
}

// Workgroup (b, sl): slice sl of bucket b's keys, counted into 2^shift LDS
// counters and written out whole to partial[(b * slices + sl) << shift ..].
// 128 KiB of LDS allows one workgroup per CU, so it has 16 waves to keep
// enough key loads in flight.
constexpr int kCountTB = 1024;

__global__ __launch_bounds__(kCountTB) void k_bucket_count(const uint32_t *__restrict__ keys,
                                                      const int32_t *__restrict__ off, int64_t ntiles,
                                                      int shift, int slices,
                                                      uint32_t *__restrict__ partial)
{
    extern __shared__ uint32_t lw[];
    const int words = 1 << shift;
    const int b = blockIdx.x / slices, sl = blockIdx.x % slices;
    for (int j = threadIdx.x; j < words; j += kCountTB) lw[j] = 0;
    __syncthreads();
    const int64_t b0 = off[(int64_t)b * ntiles], b1 = off[(int64_t)(b + 1) * ntiles];
    const int64_t per = (b1 - b0 + slices - 1) / slices;
    const int64_t k0 = b0 + sl * per, k1 = k0 + per < b1 ? k0 + per : b1;
    const uint32_t kbase = (uint32_t)b << shift;
    constexpr int U = 8;  // key loads in flight per thread
    for (int64_t kb = k0 + threadIdx.x; kb < k1; kb += U * kCountTB) {
        uint32_t v[U];
#pragma unroll
        for (int u = 0; u < U; u++) v[u] = kb + u * kCountTB < k1 ? keys[kb + u * kCountTB] - kbase : ~0u;
#pragma unroll
        for (int u = 0; u < U; u++)
            if (v[u] != ~0u) atomicAdd(&lw[v[u]], 1u);
    }
    __syncthreads();
    uint32_t *out = partial + (int64_t)blockIdx.x * words;
    for (int j = threadIdx.x; j < words; j += kCountTB) out[j] = lw[j];
}

// out[c] for c < n: the sum of counter c over the slices.
__global__ __launch_bounds__(kTB) void k_bucket_reduce(const uint32_t *__restrict__ partial, int64_t n,
                                                       int shift, int slices, uint32_t *__restrict__ out)
{
    const int64_t W = 1ll << shift;
    for (int64_t c = (int64_t)blockIdx.x * kTB + threadIdx.x; c < n; c += (int64_t)gridDim.x * kTB) {
        const int64_t b = c >> shift, j = c & (W - 1);
        uint32_t acc = 0;
        for (int s = 0; s < slices; s++) acc += partial[(b * slices + s) * W + j];
        out[c] = acc;
    }
}

// Statistics of a count sequence cnt[i] = (ptr ? ptr[i+1]-ptr[i] : vals[i]):
// sum of squares, sum of adjacent absolute differences, max, min.  Each
// workgroup reduces its share and writes one partial record; a one-workgroup
// grid writes the final fields of *acc itself, otherwise k_stats_final
// combines the partials (many atomics on one record would queue up).
struct StatPart {
    unsigned long long s2, bn;
    int mx, mn;
};

__device__ __forceinline__ void store_stats(FeatAcc *acc, int is_row, const StatPart &p)
{
    if (is_row) {
        acc->s2r = p.s2;
        acc->bnr = p.bn;
        acc->maxr = p.mx;
        acc->minr = p.mn;
    } else {
        acc->s2c = p.s2;
        acc->bnc = p.bn;
        acc->maxc = p.mx;
        acc->minc = p.mn;
    }
}

__global__ __launch_bounds__(kTB) void k_count_stats(const int32_t *__restrict__ ptr,
                                                     const int32_t *__restrict__ vals, int64_t n,
                                                     int is_row, FeatAcc *__restrict__ acc,
                                                     StatPart *__restrict__ part)
{
    __shared__ unsigned long long t64[kTB / kWave];
    __shared__ int t32[kTB / kWave];
    unsigned long long s2 = 0, bn = 0;
    int mx = 0, mn = INT_MAX;
    for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kTB) {
        int c = ptr ? ptr[i + 1] - ptr[i] : vals[i];
        s2 += (unsigned long long)c * (unsigned long long)c;
        mx = c > mx ? c : mx;
        mn = c < mn ? c : mn;
        if (i + 1 < n) {
            int c1 = ptr ? ptr[i + 2] - ptr[i + 1] : vals[i + 1];
            bn += (unsigned long long)(c1 > c ? c1 - c : c - c1);
        }
    }
    StatPart p;
    p.s2 = block_sum_u64<kTB>(s2, t64);
    p.bn = block_sum_u64<kTB>(bn, t64);
    p.mx = block_max_i32<kTB>(mx, t32);
    p.mn = block_min_i32<kTB>(mn, t32);
    if (threadIdx.x != 0) return;
    if (gridDim.x == 1)
        store_stats(acc, is_row, p);
    else
        part[blockIdx.x] = p;
}

__global__ __launch_bounds__(kTB) void k_stats_final(const StatPart *__restrict__ part, int64_t G,
                                                     int is_row, FeatAcc *__restrict__ acc)
{
    __shared__ unsigned long long t64[kTB / kWave];
    __shared__ int t32[kTB / kWave];
    unsigned long long s2 = 0, bn = 0;
    int mx = 0, mn = INT_MAX;
    for (int64_t g = threadIdx.x; g < G; g += kTB) {
        const StatPart q = part[g];
        s2 += q.s2;
        bn += q.bn;
        mx = q.mx > mx ? q.mx : mx;
        mn = q.mn < mn ? q.mn : mn;
    }
    StatPart p;
    p.s2 = block_sum_u64<kTB>(s2, t64);
    p.bn = block_sum_u64<kTB>(bn, t64);
    p.mx = block_max_i32<kTB>(mx, t32);
    p.mn = block_min_i32<kTB>(mn, t32);
    if (threadIdx.x == 0) store_stats(acc, is_row, p);
}

inline unsigned stats_grid(int64_t n)
{
    int64_t g = ceil_div(n, (int64_t)kTB * 4);
    return (unsigned)(g < 1 ? 1 : g > 2048 ? 2048 : g);
}

// Statistics of n counts into the row (is_row) or column fields of *acc.
void count_stats(const int32_t *ptr, const int32_t *vals, int64_t n, int is_row, FeatAcc *acc, hipStream_t s)
{
    const unsigned G = stats_grid(n);
    DevBuf part;
    if (G > 1) part.alloc(sizeof(StatPart) * G, s);
    k_count_stats<<<G, kTB, 0, s>>>(ptr, vals, n, is_row, acc, part.as<StatPart>());
    GS_HIP(hipGetLastError());
    if (G > 1) {
        k_stats_final<<<1, kTB, 0, s>>>(part.as<StatPart>(), G, is_row, acc);
        GS_HIP(hipGetLastError());
    }
}

// Diagonal occupancy bitmap: bit (col - row + R - 1) is set for every entry.
//
// Small spans (the bitmap and a row_ptr slice fit in one workgroup's LDS):
// workgroup p owns a contiguous range of rows, marks its entries' diagonals
// in a private LDS bitmap (one thread per entry, its row found by binary
// search in the LDS copy of the range's row_ptr slice), and writes the
// bitmap out whole; k_diag_or then ORs the per-workgroup bitmaps word by
// word.  No global atomics.
//
// Large spans: one wavefront per row marks a global bitmap with atomicOr,
// skipping the atomic when the bit is already set (bits only ever get set,
// and the main diagonal alone gets one hit per row).
constexpr int64_t kDiagLdsRows = 2048;    // rows per workgroup (8 KiB row_ptr slice)
constexpr int kDiagParts = 256;           // workgroups (partial bitmaps)
constexpr int kDiagTB = 1024;             // 16 waves per workgroup hide the gather latency

__global__ __launch_bounds__(kDiagTB) void k_diag_lds(const int32_t *__restrict__ rp,
                                                  const int32_t *__restrict__ col, int64_t R,
                                                  int64_t nw, int64_t rows_per,
                                                  uint32_t *__restrict__ partial)
{
    extern __shared__ uint32_t sm[];
    uint32_t *lbm = sm;
    int32_t *lrp = reinterpret_cast<int32_t *>(sm + nw);
    const int64_t r0 = (int64_t)blockIdx.x * rows_per < R ? (int64_t)blockIdx.x * rows_per : R;
    const int64_t r1 = r0 + rows_per < R ? r0 + rows_per : R;
    const int nr = (int)(r1 - r0);
    for (int64_t w = threadIdx.x; w < nw; w += kDiagTB) lbm[w] = 0;
    for (int i = threadIdx.x; i <= nr; i += kDiagTB) lrp[i] = rp[r0 + i];
    __syncthreads();
    const int64_t k0 = lrp[0], k1 = lrp[nr];
    constexpr int U = 4;  // column loads in flight per thread
    for (int64_t kb = k0 + threadIdx.x; kb < k1; kb += U * kDiagTB) {
        int c[U];
#pragma unroll
        for (int u = 0; u < U; u++) c[u] = kb + u * kDiagTB < k1 ? col[kb + u * kDiagTB] : 0;
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t k = kb + u * kDiagTB;
            if (k >= k1) break;
            // last row i of the range with lrp[i] <= k (empty rows share their start)
            int lo = 0, hi = nr - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (lrp[mid] <= k)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            const int64_t sidx = (int64_t)c[u] - (r0 + lo) + R - 1;
            const uint32_t bit = 1u << (sidx & 31);
            if (!(lbm[sidx >> 5] & bit)) atomicOr(&lbm[sidx >> 5], bit);
        }
    }
    __syncthreads();
    uint32_t *out = partial + (int64_t)blockIdx.x * nw;
    for (int64_t w = threadIdx.x; w < nw; w += kDiagTB) out[w] = lbm[w];
}

// Block of 1024 threads = 64 words x 16 slices of the partial bitmaps.
__global__ __launch_bounds__(1024) void k_diag_or(const uint32_t *__restrict__ partial, int64_t P,
                                                  int64_t nw, uint32_t *__restrict__ bm)
{
    __shared__ uint32_t red[16][64];
    const int lane = threadIdx.x % 64, sl = threadIdx.x / 64;
    const int64_t w = (int64_t)blockIdx.x * 64 + lane;
    uint32_t v = 0;
    if (w < nw)
        for (int64_t p = sl; p < P; p += 16) v |= partial[p * nw + w];
    red[sl][lane] = v;
    __syncthreads();
    if (sl == 0 && w < nw) {
        for (int q = 1; q < 16; q++) v |= red[q][lane];
        bm[w] = v;
    }
}

__global__ __launch_bounds__(kTB) void k_mark_diags(const int32_t *__restrict__ rp,
                                                    const int32_t *__restrict__ col, int64_t R,
                                                    uint32_t *__restrict__ bm)
{
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kTB / kWave);
    constexpr int U = 8;  // entries in flight per lane (a hub row is one wave's work)
    for (int64_t i = ((int64_t)blockIdx.x * kTB + threadIdx.x) / kWave; i < R; i += waves) {
        const int64_t e = rp[i + 1];
        for (int64_t kb = rp[i] + lane; kb < e; kb += U * kWave) {
            int64_t sidx[U];
#pragma unroll
            for (int u = 0; u < U; u++)
                sidx[u] = kb + u * kWave < e ? (int64_t)col[kb + u * kWave] - i + R - 1 : -1;
            uint32_t seen[U];
#pragma unroll
            for (int u = 0; u < U; u++)
                // the check may read a stale copy cached near this workgroup:
                // then the (idempotent) atomic is simply issued
                seen[u] = sidx[u] < 0 ? ~0u
                                      : __hip_atomic_load(&bm[sidx[u] >> 5], __ATOMIC_RELAXED,
                                                          __HIP_MEMORY_SCOPE_WORKGROUP);
#pragma unroll
            for (int u = 0; u < U; u++) {
                if (sidx[u] < 0) continue;
                const uint32_t bit = 1u << (sidx[u] & 31);
                if (!(seen[u] & bit)) atomicOr(&bm[sidx[u] >> 5], bit);
            }
        }
    }
}

// Wide spans: the bitmap in windows of `ww` words that fit in LDS.
// Workgroup (x, y) takes rows [x rows_per, (x+1) rows_per) and window y
// (bits [y 32 ww, (y+1) 32 ww) of the bitmap).  Its waves take blocks of 64
// consecutive rows in turn: the block's entries are contiguous, so all 64
// lanes walk them together, eight column loads in flight per lane, each
// finding its entry's row in the block's 65 row pointers (kept in the wave's
// LDS: a binary search for the first entry, then forward steps), and mark
// the entries whose diagonal falls in the window.  The LDS window is then
// written out as this workgroup's partial; k_diag_win_or ORs the partials of
// each window.  Every entry is read once per window; no global atomics.
// (Measured at 52M entries and 4 windows: 652 us; 748 us with one column
// load per lane, 1194 us for the global bitmap; one lane group per row
// measured 1050-1110 us: the row pointer loads then chain per row.)
constexpr int kWinRows = 64;  // rows per wave block

__global__ __launch_bounds__(kDiagTB) void k_diag_win(const int32_t *__restrict__ rp,
                                                      const int32_t *__restrict__ col, int64_t R,
                                                      int64_t nw, int64_t ww, int64_t rows_per,
                                                      uint32_t *__restrict__ partial)
{
    extern __shared__ uint32_t lbm[];
    __shared__ int32_t lrp[kDiagTB / kWave][kWinRows + 1];
    const int64_t r0 = (int64_t)blockIdx.x * rows_per < R ? (int64_t)blockIdx.x * rows_per : R;
    const int64_t r1 = r0 + rows_per < R ? r0 + rows_per : R;
    const int64_t w0 = (int64_t)blockIdx.y * ww;
    const int64_t wn = nw - w0 < ww ? nw - w0 : ww;  // words of this window
    const int64_t b0 = w0 * 32, b1 = (w0 + wn) * 32;
    for (int64_t w = threadIdx.x; w < wn; w += kDiagTB) lbm[w] = 0;
    __syncthreads();
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    int32_t *wrp = lrp[wave];
    for (int64_t i0 = r0 + (int64_t)wave * kWinRows; i0 < r1; i0 += (int64_t)(kDiagTB / kWave) * kWinRows) {
        const int nr = r1 - i0 < kWinRows ? (int)(r1 - i0) : kWinRows;
        wrp[lane] = lane <= nr ? rp[i0 + lane] : 0;
        if (lane == 0) wrp[kWinRows] = rp[i0 + nr];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const int64_t k0 = wrp[0], k1 = wrp[kWinRows];
        int lo = 0;  // row j of the block holding entry k: the last j with wrp[j] <= k
        if (k0 + lane < k1) {
            int hi = nr - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (wrp[mid] <= k0 + lane)
                    lo = mid;
                else
                    hi = mid - 1;
            }
        }
        // eight column loads in flight per lane; k grows by one wave per
        // entry, so the row is found by walking forward from the last one
        constexpr int U = 8;
        for (int64_t kb = k0 + lane; kb < k1; kb += U * kWave) {
            int c[U];  // clamped indices: the loads need no branch, so all are in flight at once
#pragma unroll
            for (int u = 0; u < U; u++) c[u] = col[kb + u * kWave < k1 ? kb + u * kWave : k1 - 1];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int64_t k = kb + u * kWave;
                if (k >= k1) break;
                while (lo < nr - 1 && wrp[lo + 1] <= k) lo++;
                const int64_t sidx = (int64_t)c[u] - (i0 + lo) + R - 1;
                if (sidx < b0 || sidx >= b1) continue;
                const int64_t b = sidx - b0;
                const uint32_t bit = 1u << (b & 31);
                if (!(lbm[b >> 5] & bit)) atomicOr(&lbm[b >> 5], bit);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();  // wrp is rewritten by the next block
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    __syncthreads();
    uint32_t *out = partial + ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * ww;
    for (int64_t w = threadIdx.x; w < wn; w += kDiagTB) out[w] = lbm[w];
}

// bm[w] = OR over the row chunks of window w / ww's partial word w % ww.
__global__ __launch_bounds__(kTB) void k_diag_win_or(const uint32_t *__restrict__ partial, int64_t nw,
                                                     int64_t ww, int64_t chunks, uint32_t *__restrict__ bm)
{
    for (int64_t w = (int64_t)blockIdx.x * kTB + threadIdx.x; w < nw; w += (int64_t)gridDim.x * kTB) {
        const int64_t y = w / ww, o = w - y * ww;
        const uint32_t *p = partial + y * chunks * ww + o;
        uint32_t v = 0;
        for (int64_t c = 0; c < chunks; c++) v |= p[c * ww];
        bm[w] = v;
    }
}

// Population count of the bitmap: one partial per workgroup (or the total
// itself, added to *total, from a one-workgroup grid).
__global__ __launch_bounds__(kTB) void k_popc_total(const uint32_t *__restrict__ bm, int64_t nw,
                                                    unsigned long long *__restrict__ part,
                                                    unsigned long long *__restrict__ total)
{
    __shared__ unsigned long long t64[kTB / kWave];
    unsigned long long s = 0;
    for (int64_t w = (int64_t)blockIdx.x * kTB + threadIdx.x; w < nw;
         w += (int64_t)gridDim.x * kTB)
        s += __popc(bm[w]);
    s = block_sum_u64<kTB>(s, t64);
    if (threadIdx.x != 0) return;
    if (gridDim.x == 1)
        *total += s;
    else
        part[blockIdx.x] = s;
}

}  // namespace

namespace {

// Column-count buckets of 2^shift columns: 32768 counters (128 KiB of LDS),
// fewer where LDS is smaller.
int bucket_shift()
{
    int w = 15;
    while (w > 10 && ((int64_t)4 << w) > max_lds_bytes()) w--;
    return w;
}

}  // namespace

void diag_bitmap(const int32_t *rp, const int32_t *col, int64_t R, int64_t C, int64_t Z,
                 uint32_t *bm, hipStream_t s)
{
    const int64_t nw = (R > 0 && C > 0) ? ceil_div(R + C - 1, 32) : 0;
    if (nw == 0) return;
    const int64_t P = std::min<int64_t>(kDiagParts, R);
    const int64_t rows_per = ceil_div(R, P);
    const char *force_ww = std::getenv("GS_DIAG_WIN_WORDS");  // tests: the windowed path with small windows
    if (Z > 0 && (nw + rows_per + 1) * 4 <= max_lds_bytes() && rows_per <= kDiagLdsRows &&
        std::getenv("GS_DIAG_GLOBAL") == nullptr && !(force_ww && *force_ww)) {
        DevBuf part;
        part.alloc((size_t)(P * nw) * 4, s);
        const size_t lds = (size_t)(nw + rows_per + 1) * 4;
        k_diag_lds<<<(unsigned)P, kDiagTB, lds, s>>>(rp, col, R, nw, rows_per, part.as<uint32_t>());
        GS_HIP(hipGetLastError());
        k_diag_or<<<(unsigned)ceil_div(nw, 64), 1024, 0, s>>>(part.as<uint32_t>(), P, nw, bm);
        GS_HIP(hipGetLastError());
        return;
    }
    if (Z > 0 && std::getenv("GS_DIAG_GLOBAL") == nullptr) {
        // windows of the bitmap that fit in LDS, about 256 workgroups in all
        int64_t ww = std::min<int64_t>(nw, (max_lds_bytes() - 8192) / 4);  // beside the waves' row pointers
        if (force_ww && *force_ww) ww = std::max<int64_t>(1, std::min<int64_t>(ww, std::atoll(force_ww)));
        const int64_t windows = ceil_div(nw, ww);
        const int64_t chunks = std::max<int64_t>(1, std::min<int64_t>(ceil_div(R, 64), ceil_div(256, windows)));
        const int64_t rows_per = ceil_div(R, chunks);
        DevBuf part;
        part.alloc((size_t)(windows * chunks * ww) * 4, s);
        k_diag_win<<<dim3((unsigned)chunks, (unsigned)windows), kDiagTB, (size_t)ww * 4, s>>>(
            rp, col, R, nw, ww, rows_per, part.as<uint32_t>());
        GS_HIP(hipGetLastError());
        k_diag_win_or<<<elem_grid(nw), kTB, 0, s>>>(part.as<uint32_t>(), nw, ww, chunks, bm);
        GS_HIP(hipGetLastError());
        return;
    }
    GS_HIP(hipMemsetAsync(bm, 0, (size_t)nw * 4, s));
    if (Z > 0) {
        k_mark_diags<<<elem_grid(R * kWave), kTB, 0, s>>>(rp, col, R, bm);
        GS_HIP(hipGetLastError());
    }
}

// Column counts cc[0..C) (cleared here).  Bucketed LDS counting when the
// matrix is large enough to pay for the extra passes, atomics otherwise.
void column_counts(const int32_t *col, int64_t C, int64_t Z, int32_t *cc, hipStream_t s)
{
    const int shift = bucket_shift();
    const int64_t nb = ceil_div(C, 1ll << shift);
    if (Z < (1 << 20) || nb > 256 || std::getenv("GS_COLHIST_ATOMIC") != nullptr) {
        GS_HIP(hipMemsetAsync(cc, 0, (size_t)C * 4, s));
        if (Z > 0) {
            k_col_hist<<<elem_grid(Z), kTB, 0, s>>>(col, Z, cc);
            GS_HIP(hipGetLastError());
        }
        return;
    }
    const uint32_t *keys = reinterpret_cast<const uint32_t *>(col);
    const int64_t ntiles = ceil_div(Z, (int64_t)kBucketTile);
    // about 512 workgroups in all (one at a time per CU at 128 KiB of LDS)
    const int slices = (int)std::max<int64_t>(1, std::min<int64_t>(64, ceil_div(512, nb)));
    DevBuf hist, sorted, partial;
    hist.alloc((size_t)(nb * ntiles + 1) * 4, s);
    sorted.alloc((size_t)Z * 4, s);
    partial.alloc(((size_t)(nb * slices) << shift) * 4, s);
    k_bucket_hist<<<(unsigned)ntiles, kTB, 0, s>>>(keys, Z, shift, (int)nb, ntiles, hist.as<int32_t>());
    GS_HIP(hipGetLastError());
    exclusive_scan_i32(hist.as<int32_t>(), hist.as<int32_t>(), nb * ntiles, true, s);
    k_bucket_scatter<<<(unsigned)ntiles, kTB, 0, s>>>(keys, Z, shift, (int)nb, ntiles, hist.as<int32_t>(),
                                                      sorted.as<uint32_t>());
    GS_HIP(hipGetLastError());
    k_bucket_count<<<(unsigned)(nb * slices), kCountTB, (size_t)4 << shift, s>>>(
        sorted.as<uint32_t>(), hist.as<int32_t>(), ntiles, shift, slices, partial.as<uint32_t>());
    GS_HIP(hipGetLastError());
    k_bucket_reduce<<<elem_grid(C), kTB, 0, s>>>(partial.as<uint32_t>(), C, shift, slices,
                                                 reinterpret_cast<uint32_t *>(cc));
    GS_HIP(hipGetLastError());
}

void features_from_csr(gs_matrix_ &csr, hipStream_t s, gs_features *out)
{
    const int64_t R = csr.R, C = csr.C, Z = csr.Z;
    const int32_t *rp = csr.row_ptr.as<int32_t>();
    const int32_t *col = csr.col.as<int32_t>();

    // every aggregate lands in one device record, read back once
    struct Out {
        FeatAcc acc;
        unsigned long long nd, nb16;
    } o = {{0, 0, 0, 0, 0, INT_MAX, 0, INT_MAX}, 0, 0};
    DevBuf d, cc, bm;
    d.alloc(sizeof(Out), s);
    GS_HIP(hipMemcpyAsync(d.p, &o, sizeof o, hipMemcpyHostToDevice, s));
    Out *dout = d.as<Out>();
    if (R > 0) {
        count_stats(rp, nullptr, R, 1, &dout->acc, s);
    }
    if (C > 0) {
        cc.alloc((size_t)C * 4, s);
        column_counts(col, C, Z, cc.as<int32_t>(), s);
        count_stats(nullptr, cc.as<int32_t>(), C, 0, &dout->acc, s);
    }
    if (Z > 0) {
        const int64_t nw = ceil_div(R + C - 1, 32);
        bm.alloc((size_t)nw * 4, s);
        diag_bitmap(rp, col, R, C, Z, bm.as<uint32_t>(), s);
        const unsigned G = stats_grid(nw);
        DevBuf part;
        if (G > 1) part.alloc(sizeof(unsigned long long) * G, s);
        k_popc_total<<<G, kTB, 0, s>>>(bm.as<uint32_t>(), nw, part.as<unsigned long long>(), &dout->nd);
        GS_HIP(hipGetLastError());
        if (G > 1) add_partials_u64(part.as<unsigned long long>(), G, &dout->nd, s);
    }
    count_blocks_async(csr, 16, &dout->nb16, s);
    GS_HIP(hipMemcpyAsync(&o, d.p, sizeof o, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));
    // a CSR handle not yet planned keeps its column counts for the plan's
    // reference classes (the selector plans the handle it extracted from)
    if (!csr.csr_planned && cc.p) csr.col_counts = std::move(cc);
    const FeatAcc &h = o.acc;
    const unsigned long long nd = o.nd;
    const int64_t nb16 = (int64_t)o.nb16;

    gs_features &f = *out;
    f.n_rows = R;
    f.n_cols = C;
    f.nnz = Z;
    f.n_diags = (int64_t)nd;
    f.max_rd = R > 0 ? h.maxr : 0;
    f.min_rd = R > 0 ? h.minr : 0;
    f.max_cd = C > 0 ? h.maxc : 0;
    f.min_cd = C > 0 ? h.minc : 0;
    f.sum_rd2 = h.s2r;
    f.sum_cd2 = h.s2c;
    f.bounce_r = h.bnr;
    f.bounce_c = h.bnc;
    f.n_blocks16 = nb16;

    finish_features(&f);
}

}  // namespace gs
