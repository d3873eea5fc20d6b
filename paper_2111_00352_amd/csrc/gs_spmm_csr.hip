// CSR SpMM, vectorised path (F a multiple of 4, 16-byte aligned operands).
//
// Work is cut at plan time into three tiers by row length:
//  * short rows (at most `long_thr` entries): one group of G lanes per row;
//    for skewed lengths (power-law graphs) ordered by decreasing length, so
//    a wavefront's groups have equal trip counts and the longest start first,
//    otherwise in natural order (neighbouring rows share X rows in L2);
//  * medium rows (up to `wg_thr` entries): one workgroup per row; its groups
//    take interleaved chunks of `chunk` entries, each summed in fresh
//    registers, and the groups' partial rows are added in LDS in group order;
//  * huge rows: chunks spread over many workgroups as independent items whose
//    partial sums a second, small launch adds in slot order.
// Every sequential fp32 chain stays within `chunk` terms and every combine
// runs in a fixed order, so results are deterministic.
//
// Lane layout: lane l of a group holds float4 q at column c0 + 4*G*q, so one
// load instruction reads G*16 contiguous bytes of an X row.  Entries are
// fetched G at a time (one per lane) and broadcast by shuffles; X rows are
// gathered several at a time (8 float4 loads in flight per lane) before any
// is consumed; the last batch of a row is masked with a select.  The grid is
// persistent (a few workgroups per CU), long-row tiles first.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <numeric>
#include <string>
#include <vector>

#include "gs_device.h"
#include "gs_gather.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kBlock = 256;

// Candidate row tiles of the LDS-staged kernel: 32 << k rows, k < kWinCands,
// each with halo 0 and 1.
constexpr int kWinCands = 4;

// Accumulates the entries [k0, k1) of one row into acc (NQ float4 per lane).
// CLS: col holds class-tagged column words (see gather_batch).
template <int NQ, int G, int U, bool CLS>
__device__ __forceinline__ void gather_entries(const int32_t *__restrict__ col,
                                               const float *__restrict__ val, int64_t k0,
                                               int64_t k1, const float *__restrict__ X,
                                               int64_t ldx, int64_t c0, const bool *qok,
                                               float *acc, int lane, int hot_cls)
{
    for (int64_t kb = k0; kb < k1; kb += G) {
        const int m = (k1 - kb) < G ? (int)(k1 - kb) : G;
        int cj = 0;
        float vj = 0.0f;
        if (lane < m) {
            cj = ld_stream(col + kb + lane);
            vj = ld_stream(val + kb + lane);
        }
        int j = 0;
        for (; j + U <= m; j += U)
            gather_batch<U, NQ, G, false, CLS>(cj, vj, j, m, X, ldx, c0, qok, acc, hot_cls);
        if (j < m) {
            if (U > 1 && m - j <= U / 2)
                gather_batch<(U > 1 ? U / 2 : 1), NQ, G, true, CLS>(cj, vj, j, m, X, ldx, c0, qok, acc, hot_cls);
            else
                gather_batch<U, NQ, G, true, CLS>(cj, vj, j, m, X, ldx, c0, qok, acc, hot_cls);
        }
    }
}

// GROUPED: the plan's group tier is active, so short items may be rows of up
// to the group limit, summed chunk by chunk (compiled out otherwise).
template <int CPL, int G, bool FULL, bool CLS, bool GROUPED>
__global__ __launch_bounds__(kBlock) void k_csr_rows(
    int64_t n_long, const int32_t *__restrict__ long_rows, const int32_t *__restrict__ rp,
    int chunk, int64_t n_short, const int4 *__restrict__ items, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ X, int64_t ldx, float *__restrict__ Y,
    int64_t ldy, int64_t F, float *__restrict__ work, int hot_cls)
{
    constexpr int GPB = kBlock / G;
    constexpr int NQ = CPL / 4;
    constexpr int U0 = 32 / CPL > 0 ? 32 / CPL : 1;  // 8 float4 loads in flight per lane
    constexpr int U = U0 < G ? U0 : G;
    __shared__ float4 part[GPB][G * NQ];
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t c0 = (int64_t)blockIdx.y * (G * CPL) + (int64_t)lane * 4;
    bool qok[NQ];
#pragma unroll
    for (int q = 0; q < NQ; q++) qok[q] = FULL || (c0 + 4 * G * q < F);
    const int64_t tiles = n_long + (n_short + GPB - 1) / GPB;

    for (int64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
        float acc[CPL];
#pragma unroll
        for (int i = 0; i < CPL; i++) acc[i] = 0.0f;
        if (t < n_long) {  // workgroup-uniform branch: one long row for all groups
            const int64_t row = long_rows[t];
            const int64_t s = rp[row], e = rp[row + 1];
            for (int64_t cs = s + (int64_t)g * chunk; cs < e; cs += (int64_t)GPB * chunk) {
                float part_acc[CPL];
#pragma unroll
                for (int i = 0; i < CPL; i++) part_acc[i] = 0.0f;
                const int64_t ce = cs + chunk < e ? cs + chunk : e;
                gather_entries<NQ, G, U, CLS>(col, val, cs, ce, X, ldx, c0, qok, part_acc, lane, hot_cls);
#pragma unroll
                for (int i = 0; i < CPL; i++) acc[i] += part_acc[i];
            }
#pragma unroll
            for (int q = 0; q < NQ; q++)
                part[g][q * G + lane] = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
            __syncthreads();
            if (g == 0) {
#pragma unroll
                for (int q = 0; q < NQ; q++) {
                    float4 a = part[0][q * G + lane];
                    for (int gg = 1; gg < GPB; gg++) {
                        const float4 b = part[gg][q * G + lane];
                        a.x += b.x;
                        a.y += b.y;
                        a.z += b.z;
                        a.w += b.w;
                    }
                    acc[4 * q] = a.x;
                    acc[4 * q + 1] = a.y;
                    acc[4 * q + 2] = a.z;
                    acc[4 * q + 3] = a.w;
                }
                store_row_stream<NQ, G>(Y + row * ldy + c0, qok, acc);
            }
            __syncthreads();  // part[] is reused by the next long row
        } else {
            const int64_t it = (t - n_long) * GPB + g;
            if (it >= n_short) break;  // later tiles of this workgroup are past the end too
            const int4 d = items[it];
            if (!GROUPED || d.z <= chunk) {
                gather_entries<NQ, G, U, CLS>(col, val, d.y, (int64_t)d.y + d.z, X, ldx, c0, qok, acc, lane,
                                              hot_cls);
            } else {  // a row of up to the group limit: chunk by chunk, each summed in fresh registers
                const int64_t e = (int64_t)d.y + d.z;
                for (int64_t cs = d.y; cs < e; cs += chunk) {
                    float part_acc[CPL];
#pragma unroll
                    for (int i = 0; i < CPL; i++) part_acc[i] = 0.0f;
                    gather_entries<NQ, G, U, CLS>(col, val, cs, cs + chunk < e ? cs + chunk : e, X, ldx, c0, qok,
                                                  part_acc, lane, hot_cls);
#pragma unroll
                    for (int i = 0; i < CPL; i++) acc[i] += part_acc[i];
                }
            }
            if (d.w < 0)
                store_row_stream<NQ, G>(Y + (int64_t)d.x * ldy + c0, qok, acc);
            else  // a chunk of a huge row: its partial sum, added later in slot order
                store_row<NQ, G>(work + (int64_t)d.w * F + c0, qok, acc);
        }
    }
}

// One group per huge row: adds the row's chunk partials (consecutive slots)
// in slot order, sixteen float4 per lane in flight, and writes the row of Y.
template <int CPL, int G>
__global__ __launch_bounds__(kBlock) void k_csr_combine(const int32_t *__restrict__ rows,
                                                        const int32_t *__restrict__ first,
                                                        int64_t n, const float *__restrict__ work,
                                                        float *__restrict__ Y, int64_t ldy, int64_t F)
{
    constexpr int GPB = kBlock / G;
    constexpr int NQ = CPL / 4;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t r = (int64_t)blockIdx.x * GPB + g;
    if (r >= n) return;
    const int64_t c0 = (int64_t)blockIdx.y * (G * CPL) + (int64_t)lane * 4;
    bool qok[NQ];
#pragma unroll
    for (int q = 0; q < NQ; q++) qok[q] = c0 + 4 * G * q < F;
    float acc[CPL];
#pragma unroll
    for (int i = 0; i < CPL; i++) acc[i] = 0.0f;
    const int64_t s0 = first[r], s1 = first[r + 1];
    // B partials in flight, summed as a tree (zeros past the last) before
    // they join the running sum: a row of n chunks adds log2(B) + n / B terms
    // in sequence
    constexpr int B = NQ >= 4 ? 4 : NQ == 2 ? 8 : 16;  // 16 float4 of partials per lane
    for (int64_t sl = s0; sl < s1; sl += B) {
        float4 p[B][NQ];
#pragma unroll
        for (int u = 0; u < B; u++)
#pragma unroll
            for (int q = 0; q < NQ; q++)
                p[u][q] = (sl + u < s1 && qok[q])
                              ? *reinterpret_cast<const float4 *>(work + (sl + u) * F + c0 + 4 * G * q)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int w = 1; w < B; w <<= 1)
#pragma unroll
            for (int u = 0; u < B; u += 2 * w)
#pragma unroll
                for (int q = 0; q < NQ; q++) {
                    p[u][q].x += p[u + w][q].x;
                    p[u][q].y += p[u + w][q].y;
                    p[u][q].z += p[u + w][q].z;
                    p[u][q].w += p[u + w][q].w;
                }
#pragma unroll
        for (int q = 0; q < NQ; q++) {
            acc[4 * q] += p[0][q].x;
            acc[4 * q + 1] += p[0][q].y;
            acc[4 * q + 2] += p[0][q].z;
            acc[4 * q + 3] += p[0][q].w;
        }
    }
    store_row_stream<NQ, G>(Y + (int64_t)rows[r] * ldy + c0, qok, acc);
}

// Row tiles with their X window staged in LDS (natural row order, rows of at
// most the short-row limit).  A workgroup takes T consecutive rows [r0, r1)
// and first copies the X rows [r0 - halo, r1 + halo) of its column slice
// into LDS with coalesced loads; its groups then run the rows as the plain
// kernel does, reading every entry whose column lies in the window from LDS
// and the others from global memory.  Graphs whose edges stay mostly inside
// such tiles (communities of consecutive nodes, stencils) then gather most
// X rows once per tile instead of once per entry through L2.
template <int CPL, int G, bool FULL>
__global__ __launch_bounds__(kBlock) void k_csr_window(
    int64_t R, int64_t C, const int32_t *__restrict__ rp, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ X, int64_t ldx, float *__restrict__ Y,
    int64_t ldy, int64_t F, int T, int halo, int64_t ntiles)
{
    constexpr int GPB = kBlock / G;
    constexpr int NQ = CPL / 4;
    constexpr int RW = G * NQ;  // float4 per staged row
    constexpr int B0 = 32 / CPL > 0 ? 32 / CPL : 1;
    constexpr int B = B0 < G ? B0 : G;  // X rows in flight per batch
    extern __shared__ float4 xs[];
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
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
            float acc[CPL];  // rows hold at most the short-row limit of entries: one chain
#pragma unroll
            for (int i = 0; i < CPL; i++) acc[i] = 0.0f;
            const int64_t s = rp[r], e = rp[r + 1];
            for (int64_t kb = s; kb < e; kb += G) {
                const int m = (e - kb) < G ? (int)(e - kb) : G;
                int cj = 0;
                float vj = 0.0f;
                if (lane < m) {
                    cj = ld_stream(col + kb + lane);
                    vj = ld_stream(val + kb + lane);
                }
                for (int j = 0; j < m; j += B)
                    window_batch<B, NQ, G>(cj, vj, j, m, xs, w0, w1, lane, X, ldx, c0, qok, acc);
            }
            store_row_stream<NQ, G>(Y + r * ldy + c0, qok, acc);
        }
    }
}

int env_int(const char *name, int dflt)
{
    const char *v = std::getenv(name);
    if (!v || !*v) return dflt;
    int x = std::atoi(v);
    return x > 0 ? x : dflt;
}

}  // namespace

// ------------------------------------------------------------------ plan
//
// csr_items = [chunk items of medium long rows | chunk items of huge rows |
// short items (slot -1)]; long_rows = [medium rows | huge rows], each part in
// decreasing length, long_first[] giving each long row's first partial slot.
// The generic path runs every chunk item and combines every long row; the
// vectorised path runs medium rows a workgroup each and only the huge rows'
// chunks (combined by a second small launch).
//
// The plan is built on the device: every row gets the 64-bit key
// (group << 32 | rank) with group 0 = medium, 1 = huge, 2 = short and rank =
// maxlen - len for long rows, thr - len for short rows of a skewed matrix
// (0 otherwise); a stable radix sort on those keys gives the row order
// (natural order within equal keys), a scan of the rows' item counts gives
// each row's first item, and one kernel writes the items.  A long row's
// chunk slots are its item positions.

namespace {

struct PlanStats {
    unsigned long long sum, sum2;
    int maxlen, n_long, n_huge, n_group;
};

// Row-length statistics: one partial record per workgroup (a one-workgroup
// grid writes the result itself); k_plan_stats_final combines the partials.
__device__ __forceinline__ PlanStats block_plan_stats(unsigned long long sum, unsigned long long sum2, int mx,
                                                      int nl, int nh, int ng)
{
    __shared__ unsigned long long t64[kBlock / kWave];
    __shared__ int t32[kBlock / kWave];
    PlanStats p;
    p.sum = block_sum_u64<kBlock>(sum, t64);
    p.sum2 = block_sum_u64<kBlock>(sum2, t64);
    p.maxlen = block_max_i32<kBlock>(mx, t32);
    p.n_long = (int)block_sum_u64<kBlock>((unsigned long long)nl, t64);
    p.n_huge = (int)block_sum_u64<kBlock>((unsigned long long)nh, t64);
    p.n_group = (int)block_sum_u64<kBlock>((unsigned long long)ng, t64);
    return p;
}

__global__ __launch_bounds__(kBlock) void k_plan_stats(const int32_t *__restrict__ rp, int64_t R,
                                                       int thr, int wg_thr, int group_max,
                                                       PlanStats *__restrict__ part,
                                                       PlanStats *__restrict__ st)
{
    unsigned long long sum = 0, sum2 = 0;
    int mx = 0, nl = 0, nh = 0, ng = 0;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * kBlock) {
        const int len = rp[i + 1] - rp[i];
        sum += (unsigned long long)len;
        sum2 += (unsigned long long)len * (unsigned long long)len;
        mx = len > mx ? len : mx;
        nl += len > thr;
        nh += len > wg_thr;
        ng += len > group_max;
    }
    const PlanStats p = block_plan_stats(sum, sum2, mx, nl, nh, ng);
    if (threadIdx.x == 0) (gridDim.x == 1 ? *st : part[blockIdx.x]) = p;
}

__global__ __launch_bounds__(kBlock) void k_plan_stats_final(const PlanStats *__restrict__ part, int64_t G,
                                                             PlanStats *__restrict__ st)
{
    unsigned long long sum = 0, sum2 = 0;
    int mx = 0, nl = 0, nh = 0, ng = 0;
    for (int64_t g = threadIdx.x; g < G; g += kBlock) {
        const PlanStats q = part[g];
        sum += q.sum;
        sum2 += q.sum2;
        mx = q.maxlen > mx ? q.maxlen : mx;
        nl += q.n_long;
        nh += q.n_huge;
        ng += q.n_group;
    }
    const PlanStats p = block_plan_stats(sum, sum2, mx, nl, nh, ng);
    if (threadIdx.x == 0) *st = p;
}

// Key of row i: its group (0 medium, 1 huge, 2 short) in the bits above the
// rank, the rank (distance below the longest length, so longer rows first)
// in the low `L` bits, so that the sort needs only L + 2 bits.
__global__ __launch_bounds__(kBlock) void k_plan_keys(const int32_t *__restrict__ rp, int64_t R,
                                                      int thr, int wg_thr, int sorted, int maxlen, int L,
                                                      uint64_t *__restrict__ keys)
{
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * kBlock) {
        const int len = rp[i + 1] - rp[i];
        const uint64_t group = len > thr ? (len > wg_thr ? 1u : 0u) : 2u;
        const uint32_t rank = group < 2 ? (uint32_t)(maxlen - len) : sorted ? (uint32_t)(thr - len) : 0u;
        keys[i] = (group << L) | rank;
    }
}

__global__ __launch_bounds__(kBlock) void k_plan_count(const int32_t *__restrict__ rp,
                                                       const uint64_t *__restrict__ keys,
                                                       const uint32_t *__restrict__ perm, int64_t R,
                                                       int chunk, int L, int32_t *__restrict__ cnt)
{
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < R;
         p += (int64_t)gridDim.x * kBlock) {
        const int64_t r = perm ? perm[p] : p;
        const int len = rp[r + 1] - rp[r];
        cnt[p] = keys && (keys[p] >> L) < 2 ? (len + chunk - 1) / chunk : 1;  // no keys: every row short
    }
}

__global__ __launch_bounds__(kBlock) void k_plan_items(const int32_t *__restrict__ rp,
                                                       const uint32_t *__restrict__ perm,
                                                       const int32_t *__restrict__ off, int64_t R,
                                                       int chunk, int64_t n_long,
                                                       int4 *__restrict__ items,
                                                       int32_t *__restrict__ long_rows,
                                                       int32_t *__restrict__ long_first)
{
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < R;
         p += (int64_t)gridDim.x * kBlock) {
        const int r = perm ? (int)perm[p] : (int)p;
        const int start = rp[r], len = rp[r + 1] - start, o = off[p];
        if (p < n_long) {
            long_rows[p] = r;
            long_first[p] = o;
            for (int j = 0, c = 0; c < len; j++, c += chunk)
                items[o + j] = make_int4(r, start + c, len - c < chunk ? len - c : chunk, o + j);
        } else {
            items[o] = make_int4(r, start, len, -1);
        }
        if (p == 0) long_first[n_long] = off[n_long];
    }
}

inline unsigned plan_grid(int64_t n)
{
    int64_t g = ceil_div(n, (int64_t)kBlock);
    return (unsigned)(g < 1 ? 1 : g > 4096 ? 4096 : g);
}

inline unsigned stats_grid(int64_t n)
{
    int64_t g = ceil_div(n, (int64_t)kBlock * 4);
    return (unsigned)(g < 1 ? 1 : g > 2048 ? 2048 : g);
}

// The item counts at the three tier boundaries, gathered for one read-back.
__global__ void k_pick3(const int32_t *__restrict__ cnt, int64_t a, int64_t b, int64_t c,
                        int32_t *__restrict__ out)
{
    if (threadIdx.x == 0) {
        out[0] = cnt[a];
        out[1] = cnt[b];
        out[2] = cnt[c];
    }
}

// Reference class of a column with n entries: the bit length of n, at most 15.
__device__ __forceinline__ int col_class(int n)
{
    const int b = 32 - __clz(n);
    return b < 15 ? b : 15;
}

// Reference class of every column, one byte each (so that the tagging pass
// gathers from an array a quarter the size of the counts), and the number of
// columns per class.  The 16 bins are counted per wave by ballots (a power
// law puts most columns in two classes: LDS atomics on one bin serialised),
// and each workgroup writes its own 16 counts to part (atomics of thousands
// of workgroups on the same 16 words queued: 50 us at 2M columns);
// k_class_total adds them.
__global__ __launch_bounds__(kBlock) void k_col_classes(const int32_t *__restrict__ cc, int64_t C,
                                                        uint8_t *__restrict__ cls, int32_t *__restrict__ part)
{
    constexpr int U = 4;  // columns per lane in flight
    __shared__ int h[16];
    if (threadIdx.x < 16) h[threadIdx.x] = 0;
    __syncthreads();
    const int lane = threadIdx.x % kWave;
    const int64_t stride = (int64_t)gridDim.x * kBlock * U;
    // every lane of a wave runs the same number of rounds, so the ballots see whole waves
    for (int64_t j0 = ((int64_t)blockIdx.x * kBlock + threadIdx.x - lane) * U; j0 < C; j0 += stride) {
        int k[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t j = j0 + u * kWave + lane;
            k[u] = j < C ? cc[j] : -1;
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int64_t j = j0 + u * kWave + lane;
            if (k[u] >= 0) {
                k[u] = col_class(k[u]);
                cls[j] = (uint8_t)k[u];
            }
        }
        for (int c = 0; c < 16; c++) {
            int n = 0;
#pragma unroll
            for (int u = 0; u < U; u++) n += __popcll(__ballot(k[u] == c));
            if (lane == 0 && n) atomicAdd(&h[c], n);
        }
    }
    __syncthreads();
    if (threadIdx.x < 16) part[(int64_t)blockIdx.x * 16 + threadIdx.x] = h[threadIdx.x];
}

// hist[c] = the sum of the G workgroups' counts of class c (one workgroup;
// sixteen readers per class, each adding every sixteenth workgroup's count).
__global__ __launch_bounds__(kBlock) void k_class_total(const int32_t *__restrict__ part, int G,
                                                        int32_t *__restrict__ hist)
{
    __shared__ int h[16];
    if (threadIdx.x < 16) h[threadIdx.x] = 0;
    __syncthreads();
    const int c = threadIdx.x % 16;
    int sum = 0;
    for (int i = threadIdx.x / 16; i < G; i += kBlock / 16) sum += part[(int64_t)i * 16 + c];
    atomicAdd(&h[c], sum);
    __syncthreads();
    if (threadIdx.x < 16) hist[threadIdx.x] = h[threadIdx.x];
}

// Class-tagged copy of the column indices: col | class(col) << 27.  Sixteen
// entries per thread (four 16-byte loads and stores), so that sixteen class
// bytes are gathered at once; a scalar tail.
__global__ __launch_bounds__(kBlock) void k_tag_cols(const int32_t *__restrict__ col, int64_t Z,
                                                     const uint8_t *__restrict__ cls, int32_t *__restrict__ tagged)
{
    const int64_t nv = Z / 16;  // whole groups of sixteen
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < nv; v += stride) {
        const int4 *src = reinterpret_cast<const int4 *>(col) + v * 4;
        int4 c[4];
#pragma unroll
        for (int u = 0; u < 4; u++) c[u] = src[u];
        int t[16];
#pragma unroll
        for (int u = 0; u < 4; u++) {
            t[4 * u + 0] = cls[c[u].x];
            t[4 * u + 1] = cls[c[u].y];
            t[4 * u + 2] = cls[c[u].z];
            t[4 * u + 3] = cls[c[u].w];
        }
        int4 *dst = reinterpret_cast<int4 *>(tagged) + v * 4;
#pragma unroll
        for (int u = 0; u < 4; u++)
            dst[u] = make_int4(c[u].x | (t[4 * u + 0] << kColClassShift), c[u].y | (t[4 * u + 1] << kColClassShift),
                               c[u].z | (t[4 * u + 2] << kColClassShift), c[u].w | (t[4 * u + 3] << kColClassShift));
    }
    for (int64_t e = nv * 16 + (int64_t)blockIdx.x * kBlock + threadIdx.x; e < Z; e += stride)
        tagged[e] = col[e] | ((int)cls[col[e]] << kColClassShift);
}

// Entries whose column lies in their row's tile window, for the row tiles
// of 32 << k rows with halo 0 (counts[2k]) and halo 1 (counts[2k+1]):
// one partial set per workgroup, added into counts.
__global__ __launch_bounds__(kBlock) void k_win_counts(const int32_t *__restrict__ rp,
                                                       const int32_t *__restrict__ col, int64_t R, int64_t C,
                                                       unsigned long long *__restrict__ counts)
{
    __shared__ unsigned long long t64[kBlock / kWave];
    unsigned long long n[2 * kWinCands] = {};
    for (int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x; r < R; r += (int64_t)gridDim.x * kBlock) {
        for (int64_t k = rp[r]; k < rp[r + 1]; k++) {
            const int64_t c = col[k];
#pragma unroll
            for (int w = 0; w < kWinCands; w++) {
                const int64_t T = 32 << w;
                const int64_t b = r / T * T, top = b + T < R ? b + T : R;
                n[2 * w] += (c >= b && c < top) ? 1u : 0u;
                n[2 * w + 1] += (c >= b - 1 && c < top + 1) ? 1u : 0u;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < 2 * kWinCands; i++) {
        const unsigned long long tot = block_sum_u64<kBlock>(n[i], t64);
        if (threadIdx.x == 0 && tot) atomicAdd(&counts[i], tot);
    }
}

}  // namespace

// Locality of the row tiles: how many entries fall in their tile's window
// for each candidate tile and halo (read back), for the LDS-staged kernel.
// Counted for natural-order matrices without long rows (GS_CSR_WINDOW = off
// skips it).
void count_windows(gs_matrix_ &m, const int32_t *rp, const int32_t *col, hipStream_t s)
{
    DevBuf cnt;
    cnt.alloc(sizeof(unsigned long long) * 2 * kWinCands, s);
    GS_HIP(hipMemsetAsync(cnt.p, 0, cnt.bytes, s));
    k_win_counts<<<stats_grid(m.R), kBlock, 0, s>>>(rp, col, m.R, m.C, cnt.as<unsigned long long>());
    GS_HIP(hipGetLastError());
    unsigned long long h[2 * kWinCands];
    GS_HIP(hipMemcpyAsync(h, cnt.p, sizeof h, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));
    for (int i = 0; i < 2 * kWinCands; i++) m.win_entries[i] = (int64_t)h[i];
    m.win_counted = true;
}

void plan_windows(gs_matrix_ &m, hipStream_t s)
{
    const char *e = std::getenv("GS_CSR_WINDOW");
    if ((e && std::string(e) == "off") || m.csr_sorted || m.csr_grouped || m.n_long_rows > 0 || m.Z == 0) return;
    count_windows(m, m.row_ptr.as<int32_t>(), m.col.as<int32_t>(), s);
}

// Measured (F = 64..256): a tile pays for its staging only when most of its
// entries are inside the window and there are several tiles per resident
// workgroup.  On the mesh (about 60% inside) the staged ELL kernel took 38
// against 34 us; on the block graph (76% inside, 6,400 tiles) 217 against
// 236 us; on matrices of 10-15k rows (a few hundred tiles) the staged CSR and
// ELL kernels were about twice as slow as the plain ones (stage, barrier and
// rows in sequence on a short critical path).
bool pick_window(const gs_matrix_ &m, int64_t row_bytes, int &T, int &h)
{
    T = h = 0;
    if (!m.win_counted) return false;
    const int64_t lds_cap = std::min<int64_t>(max_lds_bytes(), (int64_t)env_int("GS_CSR_WIN_KB", 32) * 1024);
    const int64_t min_in = m.Z * env_int("GS_CSR_WIN_PCT", 65) / 100;
    const int64_t min_tiles = env_int("GS_WIN_MIN_TILES", 2 * resident_workgroups());
    int64_t best = -1;
    for (int w = 0; w < kWinCands; w++)
        for (int hh = 0; hh < 2; hh++) {
            const int64_t bytes = (int64_t)((32 << w) + 2 * hh) * row_bytes;
            const int64_t in = m.win_entries[2 * w + hh];
            if (bytes <= lds_cap && in >= min_in && in > best && ceil_div(m.R, (int64_t)(32 << w)) >= min_tiles) {
                best = in;
                T = 32 << w;
                h = hh;
            }
        }
    if (const char *e = std::getenv("GS_CSR_WIN_T"); e && *e) {  // tests and sweeps: force a tile
        const char *he = std::getenv("GS_CSR_WIN_H");
        const int t = std::atoi(e), hh = he && std::atoi(he) > 0 ? 1 : 0;
        if (t > 0 && (int64_t)(t + 2 * hh) * row_bytes <= max_lds_bytes()) {
            T = t;
            h = hh;
        }
    }
    return T > 0;
}

// Reference classes of the columns, for gathers that keep often referenced X
// rows in the caches: counts per column, each column's class (one byte) and
// the number of columns in each class (read back).  The class-tagged copy of
// the column indices is made by the first SpMM that uses the classes.  Built
// for skewed matrices (rows ordered by length; GS_CSR_HOTCOLD = on / off
// forces it) whose column count fits the 27-bit column field.
void plan_col_classes(gs_matrix_ &m, hipStream_t s)
{
    const char *e = std::getenv("GS_CSR_HOTCOLD");
    const bool on = e && *e ? std::string(e) == "on" : m.csr_sorted;
    if (!on || m.Z == 0 || m.C > kColMask + 1) {
        m.col_counts.reset();
        return;
    }
    DevBuf cc = std::move(m.col_counts), hist;  // counted by feature extraction, if it ran
    if (!cc.p) {
        cc.alloc((size_t)m.C * 4, s);
        column_counts(m.col.as<int32_t>(), m.C, m.Z, cc.as<int32_t>(), s);
    }
    const unsigned G = std::min(plan_grid(ceil_div(m.C, 4)), 512u);
    DevBuf part;
    part.alloc((size_t)G * 16 * 4, s);
    hist.alloc(16 * 4, s);
    m.col_cls.alloc((size_t)m.C, s);
    k_col_classes<<<G, kBlock, 0, s>>>(cc.as<int32_t>(), m.C, m.col_cls.as<uint8_t>(), part.as<int32_t>());
    GS_HIP(hipGetLastError());
    k_class_total<<<1, kBlock, 0, s>>>(part.as<int32_t>(), (int)G, hist.as<int32_t>());
    GS_HIP(hipGetLastError());
    int32_t h[16];
    GS_HIP(hipMemcpyAsync(h, hist.p, sizeof h, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));
    for (int c = 0; c < 16; c++) m.col_class_cols[c] = h[c];
}

void plan_csr(gs_matrix_ &m, hipStream_t s)
{
    const int thr = env_int("GS_CSR_LONG_ROW", kCsrLongRow);
    const int chunk = std::min(env_int("GS_CSR_CHUNK", kCsrChunk), thr);
    const int wg_thr = env_int("GS_CSR_WG_ROW", kCsrWgRow);
    m.csr_long_thr = thr;
    m.csr_chunk = chunk;
    const int64_t R = m.R;
    const int32_t *rp = m.row_ptr.as<int32_t>();

    const int group_max = std::max(env_int("GS_CSR_GROUP_ROW", kCsrGroupRow), thr);
    PlanStats st = {0, 0, 0, 0, 0, 0};
    if (R > 0) {
        const unsigned G = stats_grid(R);
        DevBuf d_st, part;
        d_st.alloc(sizeof st, s);
        if (G > 1) part.alloc(sizeof(PlanStats) * G, s);
        k_plan_stats<<<G, kBlock, 0, s>>>(rp, R, thr, wg_thr, group_max, part.as<PlanStats>(),
                                          d_st.as<PlanStats>());
        GS_HIP(hipGetLastError());
        if (G > 1) {
            k_plan_stats_final<<<1, kBlock, 0, s>>>(part.as<PlanStats>(), G, d_st.as<PlanStats>());
            GS_HIP(hipGetLastError());
        }
        GS_HIP(hipMemcpyAsync(&st, d_st.p, sizeof st, hipMemcpyDeviceToHost, s));
        GS_HIP(hipStreamSynchronize(s));
    }
    // Skewed row lengths (coefficient of variation above 1/2): order by length.
    const double mean = R ? (double)st.sum / (double)R : 0.0;
    const double var = R ? std::max(0.0, (double)st.sum2 / (double)R - mean * mean) : 0.0;
    const int force = env_int("GS_CSR_SORT", 0);  // 1: never, 2: always
    bool sorted = mean > 0 && std::sqrt(var) > 0.5 * mean;
    if (force == 1) sorted = false;
    if (force == 2) sorted = true;
    m.csr_sorted = sorted;
    // A workgroup per medium row pays off for a few hub rows running beside
    // the short ones; with more medium rows than resident workgroups they
    // would queue behind each other with most of each workgroup idle, so
    // then every long row is cut into chunk items whose partial sums a second
    // launch adds.  With many more (at least 8 per resident workgroup), every
    // row of up to group_max entries instead takes one lane group, which sums
    // it chunk by chunk in registers: the rows alone fill the groups, and no
    // partial sum goes through memory.  Measured on uniform random matrices
    // of 18-50k rows of 300-1500 entries at F = 128: 1.3-1.6x faster than
    // chunk items; with 9-13k such rows chunk items stay ahead at F = 64.
    int thr_eff = thr, wg_thr_eff = wg_thr;
    int64_t n_long = st.n_long, n_huge = st.n_huge;
    const int64_t n_medium = st.n_long - st.n_huge;
    const int64_t group_min = env_int("GS_CSR_GROUP_MIN", resident_workgroups() * 8);
    m.csr_grouped = false;
    if (n_medium > group_min && group_max > thr) {
        thr_eff = wg_thr_eff = group_max;
        n_long = n_huge = st.n_group;
        m.csr_grouped = true;
    } else if (n_medium > resident_workgroups()) {
        wg_thr_eff = thr;
        n_huge = st.n_long;
    }
    m.csr_wg_thr = wg_thr_eff;
    m.n_long_rows = n_long;
    m.n_medium_rows = n_long - n_huge;
    m.n_short = R - n_long;

    int32_t h_off[3] = {0, 0, 0};
    DevBuf ka, kb, pa, pb, cnt;
    uint32_t *perm = nullptr;
    if (R > 0) {
        // ranks are at most max(longest row, thr): L bits, the group above them
        const int L = bits_for(std::max(st.maxlen, thr_eff));
        uint64_t *keys = nullptr;
        if (sorted || n_long > 0) {  // otherwise every key is equal: natural order, no sort
            ka.alloc((size_t)R * 8, s);
            kb.alloc((size_t)R * 8, s);
            pa.alloc((size_t)R * 4, s);
            pb.alloc((size_t)R * 4, s);
            k_plan_keys<<<plan_grid(R), kBlock, 0, s>>>(rp, R, thr_eff, wg_thr_eff, sorted ? 1 : 0, st.maxlen,
                                                        L, ka.as<uint64_t>());
            GS_HIP(hipGetLastError());
            std::vector<int> shifts;
            for (int sft = 0; sft < L + 2; sft += 8) shifts.push_back(sft);
            radix_sort_pairs(ka.as<uint64_t>(), kb.as<uint64_t>(), pa.as<uint32_t>(), pb.as<uint32_t>(), R,
                             shifts, s, &keys, &perm);
        }
        cnt.alloc((size_t)(R + 1) * 4, s);
        k_plan_count<<<plan_grid(R), kBlock, 0, s>>>(rp, keys, perm, R, chunk, L, cnt.as<int32_t>());
        GS_HIP(hipGetLastError());
        exclusive_scan_i32(cnt.as<int32_t>(), cnt.as<int32_t>(), R, true, s);
        DevBuf picked;
        picked.alloc(sizeof h_off, s);
        k_pick3<<<1, kWave, 0, s>>>(cnt.as<int32_t>(), m.n_medium_rows, n_long, R, picked.as<int32_t>());
        GS_HIP(hipGetLastError());
        GS_HIP(hipMemcpyAsync(h_off, picked.p, sizeof h_off, hipMemcpyDeviceToHost, s));
        GS_HIP(hipStreamSynchronize(s));
    }
    m.n_medium_chunks = h_off[0];
    m.n_long_chunks = h_off[1];
    m.n_items = h_off[2];
    m.csr_items.alloc((size_t)m.n_items * sizeof(int4), s);
    m.long_rows.alloc((size_t)n_long * 4, s);
    m.long_first.alloc((size_t)(n_long + 1) * 4, s);
    if (R > 0) {
        k_plan_items<<<plan_grid(R), kBlock, 0, s>>>(rp, perm, cnt.as<int32_t>(), R, chunk, n_long,
                                                     m.csr_items.as<int4>(), m.long_rows.as<int32_t>(),
                                                     m.long_first.as<int32_t>());
        GS_HIP(hipGetLastError());
    } else {
        GS_HIP(hipMemsetAsync(m.long_first.p, 0, 4, s));
    }
    plan_col_classes(m, s);
    plan_windows(m, s);
    m.csr_planned = true;
}

// ------------------------------------------------------------- launcher

bool spmm_csr_vec4(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                   hipStream_t s, const WorkArea *fixed)
{
    auto al = [](const void *p) { return ((uintptr_t)p % 16) == 0; };
    if (F % 4 || ldx % 4 || ldy % 4 || !al(X) || !al(Y)) return false;
    // Lane shape, measured over 160 profiled matrices at F = 64..256: four
    // columns per lane (wide groups, 8 X rows in flight per lane) is best or
    // near it, except in natural row order for very short rows (fewer than 8
    // entries on average) and for wide X (F >= 256) with rows under 64
    // entries, where 16 columns per lane -- more rows per wave -- wins.
    const bool many_rows_per_wave =
        !m.csr_sorted && (m.Z < 8 * m.R || (F >= 256 && m.Z < 64 * m.R));
    int cpl = env_int("GS_CSR_CPL", many_rows_per_wave ? 16 : 4);
    if (cpl != 4 && cpl != 8 && cpl != 16) cpl = 16;
    while (cpl > 4 && F < 4 * (int64_t)cpl) cpl /= 2;  // at least 4 lanes per group
    const int64_t lanes = ceil_div(F, cpl);
    const int g = lanes <= 4 ? 4 : lanes <= 8 ? 8 : lanes <= 16 ? 16 : lanes <= 32 ? 32 : 64;
    const int64_t slices = ceil_div(F, (int64_t)g * cpl);
    const bool full = (F % ((int64_t)g * cpl)) == 0;
    // Reference classes: the rows of the most referenced columns, whole
    // classes of them up to GS_CSR_HOT_KB (64 MiB) at this width, are
    // gathered with plain loads, every other row non-temporally, so that
    // rows read a few times do not displace them from the memory-side cache.
    // Measured on the 2M-row power-law graph at F = 128 (52M entries, rows
    // of columns with at least 64 entries hot): 3426 -> 3126 us; budgets of
    // 4 / 32 / 128 / 256 MiB gave 4185 / 3286 / 3231 / 3306 us.  Not used
    // when the rows of every referenced column fit the budget.
    int hot_cls = 0;
    if (m.col_cls.p && cpl == 4) {
        const int64_t budget = (int64_t)env_int("GS_CSR_HOT_KB", 65536) * 1024 / (F * 4);
        int64_t cum = 0;
        for (int c = 15; c >= 1 && !hot_cls; c--) {
            cum += m.col_class_cols[c];
            if (cum > budget) hot_cls = c < 15 ? c + 1 : 15;
        }
        if (hot_cls && !m.csr_colf.p) {
            if (fixed) {
                hot_cls = 0;  // no allocation allowed: plain gathers
            } else {          // first use: the class-tagged column copy
                m.csr_colf.alloc((size_t)m.Z * 4, s);
                k_tag_cols<<<plan_grid(ceil_div(m.Z, 16)), kBlock, 0, s>>>(
                    m.col.as<int32_t>(), m.Z, m.col_cls.as<uint8_t>(), m.csr_colf.as<int32_t>());
                GS_HIP(hipGetLastError());
            }
        }
    }
    // LDS-staged row tiles (pick_window): the candidate (tile, halo) that
    // keeps the most entries in the window within GS_CSR_WIN_KB (32 KiB) of
    // LDS per workgroup.  More LDS per workgroup costs resident waves: on the
    // block-community graph (F = 256) tiles of 32 / 64 / 128 rows (32 / 64 /
    // 128 KiB) measured 193 / 280 / 480 us against 209 us without staging
    // (with today's plain kernel both take 203 us there).
    int win_T = 0, win_h = 0;
    if (m.n_long_rows == 0 && !m.csr_grouped) pick_window(m, (int64_t)g * cpl * 4, win_T, win_h);
    auto launch = [&](auto cpl_t, auto g_t, auto full_t) {
        constexpr int CPL = decltype(cpl_t)::value, G = decltype(g_t)::value;
        constexpr bool FU = decltype(full_t)::value;
        constexpr int GPB = kBlock / G;
        if (win_T > 0) {
            const int64_t ntiles = ceil_div(m.R, win_T);
            const size_t lds = (size_t)(win_T + 2 * win_h) * G * CPL * 4;
            const int64_t cap = (int64_t)resident_workgroups() * env_int("GS_WG_MULT", 8);
            dim3 grid((unsigned)std::max<int64_t>(1, std::min(ntiles, cap / slices)), (unsigned)slices);
            k_csr_window<CPL, G, FU><<<grid, kBlock, lds, s>>>(m.R, m.C, m.row_ptr.as<int32_t>(),
                                                               m.col.as<int32_t>(), m.val.as<float>(), X, ldx, Y,
                                                               ldy, F, win_T, win_h, ntiles);
            GS_HIP(hipGetLastError());
            return;
        }
        const int64_t n_group_items = m.n_items - m.n_medium_chunks;  // huge chunks + short rows
        const int64_t n_huge = m.n_long_rows - m.n_medium_rows;
        const int64_t tiles = m.n_medium_rows + ceil_div(n_group_items, GPB);
        if (!tiles) return;
        float *work = n_huge ? (float *)work_for(m, fixed, (size_t)m.n_long_chunks * F * 4, s) : nullptr;
        // persistent grid: a few resident workgroups per CU (measured: 4 for
        // length-sorted rows, 8 -- about one tile each -- for natural order)
        const int64_t cap = (int64_t)resident_workgroups() * env_int("GS_WG_MULT", m.csr_sorted ? 4 : 8);
        dim3 grid((unsigned)std::max<int64_t>(1, std::min(tiles, cap / slices)), (unsigned)slices);
        auto rows = [&](auto cls_t, auto grp_t, const int32_t *cols) {
            constexpr bool CL = decltype(cls_t)::value, GR = decltype(grp_t)::value;
            k_csr_rows<CPL, G, FU, CL, GR><<<grid, kBlock, 0, s>>>(
                m.n_medium_rows, m.long_rows.as<int32_t>(), m.row_ptr.as<int32_t>(), m.csr_chunk, n_group_items,
                m.csr_items.as<int4>() + m.n_medium_chunks, cols, m.val.as<float>(), X, ldx, Y, ldy, F, work,
                hot_cls);
            GS_HIP(hipGetLastError());
        };
        bool done = false;
        if constexpr (CPL == 4) {  // reference classes: only the length-sorted lane shape
            if (hot_cls) {
                if (m.csr_grouped)
                    rows(std::true_type{}, std::true_type{}, m.csr_colf.as<int32_t>());
                else
                    rows(std::true_type{}, std::false_type{}, m.csr_colf.as<int32_t>());
                done = true;
            }
        }
        if (!done) {
            if (m.csr_grouped)
                rows(std::false_type{}, std::true_type{}, m.col.as<int32_t>());
            else
                rows(std::false_type{}, std::false_type{}, m.col.as<int32_t>());
        }
        if (n_huge) {
            dim3 g2((unsigned)ceil_div(n_huge, GPB), (unsigned)slices);
            k_csr_combine<CPL, G><<<g2, kBlock, 0, s>>>(m.long_rows.as<int32_t>() + m.n_medium_rows,
                                                        m.long_first.as<int32_t>() + m.n_medium_rows,
                                                        n_huge, work, Y, ldy, F);
            GS_HIP(hipGetLastError());
        }
    };
#define GS_L(C, GG)                                                                                  \
    if (cpl == C && g == GG) {                                                                       \
        if (full)                                                                                    \
            launch(std::integral_constant<int, C>{}, std::integral_constant<int, GG>{}, std::true_type{}); \
        else                                                                                         \
            launch(std::integral_constant<int, C>{}, std::integral_constant<int, GG>{}, std::false_type{}); \
        return true;                                                                                 \
    }
    GS_L(16, 4) GS_L(16, 8) GS_L(16, 16) GS_L(16, 32) GS_L(16, 64)
    GS_L(8, 4) GS_L(8, 8) GS_L(8, 16) GS_L(8, 32) GS_L(8, 64)
    GS_L(4, 4) GS_L(4, 8) GS_L(4, 16) GS_L(4, 32) GS_L(4, 64)
#undef GS_L
    return false;
}

}  // namespace gs
