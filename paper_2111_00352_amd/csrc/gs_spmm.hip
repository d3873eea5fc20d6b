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
#include <cstdlib>
#include <cstring>
#include <vector>

#include "gs_device.h"
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
    Acc<VEC> acc = gather_range<VEC, G>(col, val, d.y, (int64_t)d.y + d.z, X, ldx, c0, active, lane);
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
// Segmented reduction over the (row, col)-sorted triplets.  Group q owns
// entries [bounds[q], bounds[q+1]): the whole rows that start in one window
// of CH entry positions (at most 2*CH - 1 entries), or one CH-entry piece of
// a row longer than CH.  Row boundaries inside the
// chunk are found with a ballot over "row differs from the previous entry";
// a segment is written straight to Y unless its row continues into a
// neighbouring chunk (only a split row does), in which case its partial
// goes to a carry slot: slot H (index 0) for the chunk's first segment when
// that row began in an earlier chunk, slot T (index 1) for the chunk's last
// segment when its row begins here and continues.  k_coo_fixup then adds
// each split row's carries in chunk order.

template <int VEC>
__device__ __forceinline__ void coo_flush(const Acc<VEC> &acc, int64_t row, bool first_seg,
                                          bool last_seg, bool head_cont, bool tail_cont,
                                          int64_t q, float *__restrict__ Y, int64_t ldy,
                                          float *__restrict__ work, int64_t F, int64_t c0,
                                          bool active)
{
    if (!active) return;
    if (first_seg && head_cont)
        st_vec<VEC>(work + (q * 2 + 0) * F + c0, acc.vec());
    else if (last_seg && tail_cont)
        st_vec<VEC>(work + (q * 2 + 1) * F + c0, acc.vec());
    else
        st_vec_stream<VEC>(Y + row * ldy + c0, acc.vec());
}

template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_coo_main(int64_t Z, const int32_t *__restrict__ row,
                                                     const int32_t *__restrict__ col,
                                                     const float *__restrict__ val,
                                                     const float *__restrict__ X, int64_t ldx,
                                                     float *__restrict__ Y, int64_t ldy, int64_t F,
                                                     const int32_t *__restrict__ bounds, int64_t n_chunks,
                                                     float *__restrict__ work)
{
    constexpr int GPB = kBlock / G;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * VEC) + (int64_t)lane * VEC;
    const bool active = c0 < F;
    const int64_t q = xcd_tile(blockIdx.x, gridDim.x) * GPB + g;
    if (q >= n_chunks) return;
    const int64_t k0 = bounds[q], k1 = bounds[q + 1];
    const bool head_cont = k0 > 0 && row[k0 - 1] == row[k0];
    const bool tail_cont = k1 < Z && row[k1] == row[k1 - 1];
    const int gbase = (threadIdx.x % kWave) / G * G;  // first lane of this group in the wave

    Acc<VEC> acc;
    acc.zero();
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
                    coo_flush<VEC>(acc, cur, first_seg, false, head_cont, tail_cont, q, Y, ldy,
                                   work, F, c0, active);
                    first_seg = false;
                    acc.zero();
                    cur = rs[u];
                }
                if (active) acc.fma(vs[u], xs[u]);
            }
        }
    }
    coo_flush<VEC>(acc, cur, first_seg, true, head_cont, tail_cont, q, Y, ldy, work, F, c0,
                   active);
}

// Groups [0, n_split): split row e (the int4 {row, first chunk q, piece
// count n, 0}) adds its carries in chunk order, slot T of chunk q and then
// slot H of chunks q+1 .. q+n-1, eight loads in flight, and writes Y.  The
// groups after those zero the empty rows.
template <int VEC, int G>
__global__ __launch_bounds__(kBlock) void k_coo_fixup(const int4 *__restrict__ split, int64_t n_split,
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
        const int4 d = split[e];
        const int64_t q = d.y, n = d.z;
        Acc<VEC> acc;
        acc.zero();
        for (int64_t p0 = 0; p0 < n; p0 += 8) {
            Vec<VEC> h[8];
#pragma unroll
            for (int u = 0; u < 8; u++) {
                const int64_t p = p0 + u < n ? p0 + u : n - 1;
                h[u] = ld_vec<VEC>(work + ((q + p) * 2 + (p == 0 ? 1 : 0)) * F + c0);
            }
#pragma unroll
            for (int u = 0; u < 8; u++) {
                if (p0 + u >= n) break;
#pragma unroll
                for (int i = 0; i < VEC; i++) acc.v[i] += h[u].v[i];
            }
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
        for (int64_t c = lane; c < F; c += kWave) {
            const double x = (double)X[j * ldx + c];
            for (int32_t k = k0; k < k1; k++)
                unsafeAtomicAdd(&W[(int64_t)ri[k] * F + c], (double)val[k] * x);
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
    Acc<VEC> a0, a1;
    a0.zero();
    a1.zero();
    for (int64_t kb = 0; kb < K; kb += G) {
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
    a0.add(a1);
    if (active) st_vec_stream<VEC>(Y + row * ldy + c0, a0.vec());
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
    Acc<VEC> a0, a1;
    a0.zero();
    a1.zero();
    int64_t d = 0;
    for (; d + 2 <= ND; d += 2) {
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
    a0.add(a1);
    if (active) st_vec_stream<VEC>(Y + row * ldy + c0, a0.vec());
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
    Acc<VEC> acc[RPT];
#pragma unroll
    for (int r = 0; r < RPT; r++) acc[r].zero();
    for (int64_t blk = bptr[br]; blk < bptr[br + 1]; blk++) {
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
        const int rr = g + r * RG;
        const int64_t row = br * b + rr;
        if (rr < b && row < R) st_vec_stream<VEC>(Y + row * ldy + c0, acc[r].vec());
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

int env_int_coo(const char *name, int dflt)
{
    const char *v = std::getenv(name);
    if (!v || !*v) return dflt;
    int x = std::atoi(v);
    return x > 0 ? x : dflt;
}

}  // namespace

// --------------------------------------------------------------- plans

// COO chunks follow row boundaries.  The chunk bounds are the sorted,
// de-duplicated union of (a) for every window [q*CH, (q+1)*CH) of entry
// positions, the first row start at or after q*CH, and (b) for every row
// longer than CH, its start, end and CH-entry piece boundaries.  A chunk
// then holds the whole rows that start in one window (at most 2*CH - 1
// entries, every row at most CH) or one piece of a long row, whose partial
// sums the fixup launch adds.  Also lists the split rows and the empty rows,
// which the kernel must zero.  Built on the device: counts, scans, one radix
// sort, compactions.

namespace {

constexpr int kPB = 256;

inline unsigned plan_blocks(int64_t n)
{
    int64_t g = ceil_div(n, (int64_t)kPB);
    return (unsigned)(g < 1 ? 1 : g > 8192 ? 8192 : g);
}

// Smallest i in [0, n) with a[i] >= t, or n.
__device__ __forceinline__ int64_t lower_bound_i32(const int32_t *a, int64_t n, int64_t t)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (a[mid] < t)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(kPB) void k_coo_row_counts(const int32_t *__restrict__ rp, int64_t R, int chunk,
                                                        int32_t *__restrict__ cand, int32_t *__restrict__ is_long,
                                                        int32_t *__restrict__ is_empty)
{
    for (int64_t i = (int64_t)blockIdx.x * kPB + threadIdx.x; i < R; i += (int64_t)gridDim.x * kPB) {
        const int len = rp[i + 1] - rp[i];
        const bool lg = len > chunk;
        cand[i] = lg ? (len + chunk - 1) / chunk + 1 : 0;  // start, piece boundaries, end
        is_long[i] = lg;
        is_empty[i] = len == 0;
    }
}

__global__ __launch_bounds__(kPB) void k_coo_window_cands(const int32_t *__restrict__ rp, int64_t R, int64_t Z,
                                                          int chunk, int64_t W, uint64_t *__restrict__ keys)
{
    for (int64_t q = (int64_t)blockIdx.x * kPB + threadIdx.x; q < W; q += (int64_t)gridDim.x * kPB) {
        const int64_t t = q * chunk;
        const int64_t i = t > Z ? R + 1 : lower_bound_i32(rp, R + 1, t);
        keys[q] = (uint64_t)(i <= R ? rp[i] : Z);
    }
}

__global__ __launch_bounds__(kPB) void k_coo_long_cands(const int32_t *__restrict__ rp, int64_t R, int chunk,
                                                        const int32_t *__restrict__ coff, int64_t W,
                                                        uint64_t *__restrict__ keys)
{
    for (int64_t i = (int64_t)blockIdx.x * kPB + threadIdx.x; i < R; i += (int64_t)gridDim.x * kPB) {
        const int n = coff[i + 1] - coff[i];
        const int64_t s0 = rp[i], e = rp[i + 1];
        for (int k = 0; k < n; k++) {
            const int64_t b = s0 + (int64_t)k * chunk;
            keys[W + coff[i] + k] = (uint64_t)(b < e ? b : e);
        }
    }
}

__global__ __launch_bounds__(kPB) void k_flag_new(const uint64_t *__restrict__ keys, int64_t n,
                                                  int32_t *__restrict__ flag)
{
    for (int64_t k = (int64_t)blockIdx.x * kPB + threadIdx.x; k < n; k += (int64_t)gridDim.x * kPB)
        flag[k] = k == 0 || keys[k] != keys[k - 1];
}

__global__ __launch_bounds__(kPB) void k_compact_bounds(const uint64_t *__restrict__ keys, int64_t n,
                                                        const int32_t *__restrict__ off,
                                                        int32_t *__restrict__ bounds)
{
    for (int64_t k = (int64_t)blockIdx.x * kPB + threadIdx.x; k < n; k += (int64_t)gridDim.x * kPB)
        if (off[k + 1] > off[k]) bounds[off[k]] = (int32_t)keys[k];
}

__global__ __launch_bounds__(kPB) void k_coo_lists(const int32_t *__restrict__ rp, int64_t R, int chunk,
                                                   const int32_t *__restrict__ loff,
                                                   const int32_t *__restrict__ eoff,
                                                   const int32_t *__restrict__ bounds, int64_t nbnd,
                                                   int4 *__restrict__ split, int32_t *__restrict__ empty)
{
    for (int64_t i = (int64_t)blockIdx.x * kPB + threadIdx.x; i < R; i += (int64_t)gridDim.x * kPB) {
        if (loff[i + 1] > loff[i]) {
            const int len = rp[i + 1] - rp[i];
            const int64_t first = lower_bound_i32(bounds, nbnd, rp[i]);  // rp[i] is a bound
            split[loff[i]] = make_int4((int)i, (int)first, (len + chunk - 1) / chunk, 0);
        }
        if (eoff[i + 1] > eoff[i]) empty[eoff[i]] = (int32_t)i;
    }
}

}  // namespace

void plan_coo(gs_matrix_ &m, const int32_t *row_ptr, hipStream_t s)
{
    const int chunk = env_int_coo("GS_COO_CHUNK", kCooChunk);
    m.coo_chunk = chunk;
    const int64_t R = m.R, Z = m.Z;
    DevBuf cand, lng, emp;
    cand.alloc((size_t)(R + 1) * 4, s);
    lng.alloc((size_t)(R + 1) * 4, s);
    emp.alloc((size_t)(R + 1) * 4, s);
    if (R > 0) {
        k_coo_row_counts<<<plan_blocks(R), kPB, 0, s>>>(row_ptr, R, chunk, cand.as<int32_t>(),
                                                         lng.as<int32_t>(), emp.as<int32_t>());
        GS_HIP(hipGetLastError());
    }
    exclusive_scan_i32(cand.as<int32_t>(), cand.as<int32_t>(), R, true, s);
    exclusive_scan_i32(lng.as<int32_t>(), lng.as<int32_t>(), R, true, s);
    exclusive_scan_i32(emp.as<int32_t>(), emp.as<int32_t>(), R, true, s);
    int32_t tot[3] = {0, 0, 0};
    GS_HIP(hipMemcpyAsync(&tot[0], cand.as<int32_t>() + R, 4, hipMemcpyDeviceToHost, s));
    GS_HIP(hipMemcpyAsync(&tot[1], lng.as<int32_t>() + R, 4, hipMemcpyDeviceToHost, s));
    GS_HIP(hipMemcpyAsync(&tot[2], emp.as<int32_t>() + R, 4, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));

    const int64_t W = ceil_div(Z, (int64_t)chunk) + 1;  // the last window starts at or past Z
    const int64_t n = W + tot[0];
    DevBuf ka, kb, pa, pb, flag;
    ka.alloc((size_t)n * 8, s);
    kb.alloc((size_t)n * 8, s);
    pa.alloc((size_t)n * 4, s);
    pb.alloc((size_t)n * 4, s);
    flag.alloc((size_t)(n + 1) * 4, s);
    k_coo_window_cands<<<plan_blocks(W), kPB, 0, s>>>(row_ptr, R, Z, chunk, W, ka.as<uint64_t>());
    GS_HIP(hipGetLastError());
    if (tot[0]) {
        k_coo_long_cands<<<plan_blocks(R), kPB, 0, s>>>(row_ptr, R, chunk, cand.as<int32_t>(), W,
                                                         ka.as<uint64_t>());
        GS_HIP(hipGetLastError());
    }
    std::vector<int> shifts;
    for (int sft = 0; sft < bits_for(Z); sft += 8) shifts.push_back(sft);
    uint64_t *keys = nullptr;
    uint32_t *perm = nullptr;
    radix_sort_pairs(ka.as<uint64_t>(), kb.as<uint64_t>(), pa.as<uint32_t>(), pb.as<uint32_t>(), n, shifts, s,
                     &keys, &perm);
    k_flag_new<<<plan_blocks(n), kPB, 0, s>>>(keys, n, flag.as<int32_t>());
    GS_HIP(hipGetLastError());
    exclusive_scan_i32(flag.as<int32_t>(), flag.as<int32_t>(), n, true, s);
    int32_t nbnd = 0;
    GS_HIP(hipMemcpyAsync(&nbnd, flag.as<int32_t>() + n, 4, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));

    m.n_coo_chunks = nbnd - 1;
    m.n_coo_split = tot[1];
    m.n_empty_rows = tot[2];
    m.coo_bounds.alloc((size_t)nbnd * 4, s);
    m.coo_split.alloc((size_t)tot[1] * sizeof(int4), s);
    m.empty_rows.alloc((size_t)tot[2] * 4, s);
    k_compact_bounds<<<plan_blocks(n), kPB, 0, s>>>(keys, n, flag.as<int32_t>(), m.coo_bounds.as<int32_t>());
    GS_HIP(hipGetLastError());
    if (R > 0 && (tot[1] || tot[2])) {
        k_coo_lists<<<plan_blocks(R), kPB, 0, s>>>(row_ptr, R, chunk, lng.as<int32_t>(), emp.as<int32_t>(),
                                                   m.coo_bounds.as<int32_t>(), nbnd, m.coo_split.as<int4>(),
                                                   m.empty_rows.as<int32_t>());
        GS_HIP(hipGetLastError());
    }
}

// --------------------------------------------------------------- launchers

void spmm_csr(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s)
{
    if (!m.csr_planned) plan_csr(m, s);
    if (spmm_csr_vec4(m, X, ldx, Y, ldy, F, s)) return;
    const Shape sh = pick_shape(X, ldx, Y, ldy, F);
    if (m.n_long_chunks) ensure_work(m, (size_t)m.n_long_chunks * F * 4, s);
    dispatch(sh, [&]<int VEC, int G>() {
        constexpr int GPB = kBlock / G;
        if (m.n_items) {
            dim3 grid(u32_grid(ceil_div(m.n_items, GPB)), (unsigned)sh.fslices);
            k_csr_items_generic<VEC, G><<<grid, kBlock, 0, s>>>(
                m.n_items, m.csr_items.as<int4>(), m.col.as<int32_t>(), m.val.as<float>(), X, ldx, Y,
                ldy, F, m.work.as<float>());
            GS_HIP(hipGetLastError());
        }
        if (m.n_long_rows) {
            dim3 g2(u32_grid(ceil_div(m.n_long_rows, GPB)), (unsigned)sh.fslices);
            k_csr_combine<VEC, G><<<g2, kBlock, 0, s>>>(m.long_rows.as<int32_t>(),
                                                        m.long_first.as<int32_t>(), m.n_long_rows,
                                                        m.work.as<float>(), Y, ldy, F);
            GS_HIP(hipGetLastError());
        }
    });
}

void spmm_coo(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s)
{
    const Shape sh = pick_shape(X, ldx, Y, ldy, F);
    const int64_t n_chunks = m.n_coo_chunks;
    if (m.n_coo_split) ensure_work(m, (size_t)n_chunks * 2 * F * 4, s);
    dispatch(sh, [&]<int VEC, int G>() {
        constexpr int GPB = kBlock / G;
        if (n_chunks) {
            dim3 grid(u32_grid(ceil_div(n_chunks, GPB)), (unsigned)sh.fslices);
            k_coo_main<VEC, G><<<grid, kBlock, 0, s>>>(m.Z, m.row.as<int32_t>(), m.col.as<int32_t>(),
                                                       m.val.as<float>(), X, ldx, Y, ldy, F,
                                                       m.coo_bounds.as<int32_t>(), n_chunks,
                                                       m.work.as<float>());
            GS_HIP(hipGetLastError());
        }
        const int64_t groups = m.n_coo_split + m.n_empty_rows;
        if (groups) {
            dim3 g2(u32_grid(ceil_div(groups, GPB)), (unsigned)sh.fslices);
            k_coo_fixup<VEC, G><<<g2, kBlock, 0, s>>>(m.coo_split.as<int4>(), m.n_coo_split,
                                                      m.work.as<float>(), m.empty_rows.as<int32_t>(),
                                                      m.n_empty_rows, Y, ldy, F);
            GS_HIP(hipGetLastError());
        }
    });
}

void spmm_csc(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
              hipStream_t s)
{
    const int64_t n = m.R * F;
    if (n == 0) return;
    ensure_work(m, (size_t)n * 8, s);
    double *W = m.work.as<double>();
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
