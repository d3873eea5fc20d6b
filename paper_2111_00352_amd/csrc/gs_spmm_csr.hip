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
#include <vector>

#include "gs_device.h"
#include "gs_gather.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kBlock = 256;

// Accumulates the entries [k0, k1) of one row into acc (NQ float4 per lane).
template <int NQ, int G, int U>
__device__ __forceinline__ void gather_entries(const int32_t *__restrict__ col,
                                               const float *__restrict__ val, int64_t k0,
                                               int64_t k1, const float *__restrict__ X,
                                               int64_t ldx, int64_t c0, const bool *qok,
                                               float *acc, int lane)
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
        for (; j + U <= m; j += U) gather_batch<U, NQ, G, false>(cj, vj, j, m, X, ldx, c0, qok, acc);
        if (j < m) {
            if (U > 1 && m - j <= U / 2)
                gather_batch<(U > 1 ? U / 2 : 1), NQ, G, true>(cj, vj, j, m, X, ldx, c0, qok, acc);
            else
                gather_batch<U, NQ, G, true>(cj, vj, j, m, X, ldx, c0, qok, acc);
        }
    }
}

template <int CPL, int G, bool FULL>
__global__ __launch_bounds__(kBlock) void k_csr_rows(
    int64_t n_long, const int32_t *__restrict__ long_rows, const int32_t *__restrict__ rp,
    int chunk, int64_t n_short, const int4 *__restrict__ items, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ X, int64_t ldx, float *__restrict__ Y,
    int64_t ldy, int64_t F, float *__restrict__ work)
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
                gather_entries<NQ, G, U>(col, val, cs, ce, X, ldx, c0, qok, part_acc, lane);
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
            gather_entries<NQ, G, U>(col, val, d.y, (int64_t)d.y + d.z, X, ldx, c0, qok, acc, lane);
            if (d.w < 0)
                store_row_stream<NQ, G>(Y + (int64_t)d.x * ldy + c0, qok, acc);
            else  // a chunk of a huge row: its partial sum, added later in slot order
                store_row<NQ, G>(work + (int64_t)d.w * F + c0, qok, acc);
        }
    }
}

// One group per huge row: adds the row's chunk partials (consecutive slots)
// in slot order, eight in flight, and writes the row of Y.
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
    for (int64_t sl = s0; sl < s1; sl += 8) {
        float4 p[8][NQ];
#pragma unroll
        for (int u = 0; u < 8; u++)
#pragma unroll
            for (int q = 0; q < NQ; q++)
                p[u][q] = (sl + u < s1 && qok[q])
                              ? *reinterpret_cast<const float4 *>(work + (sl + u) * F + c0 + 4 * G * q)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int u = 0; u < 8; u++)
#pragma unroll
            for (int q = 0; q < NQ; q++) {
                if (sl + u >= s1) continue;
                acc[4 * q] += p[u][q].x;
                acc[4 * q + 1] += p[u][q].y;
                acc[4 * q + 2] += p[u][q].z;
                acc[4 * q + 3] += p[u][q].w;
            }
    }
    store_row_stream<NQ, G>(Y + (int64_t)rows[r] * ldy + c0, qok, acc);
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

void plan_csr(gs_matrix_ &m, hipStream_t s)
{
    const int thr = env_int("GS_CSR_LONG_ROW", kCsrLongRow);
    const int chunk = std::min(env_int("GS_CSR_CHUNK", kCsrChunk), thr);
    m.csr_long_thr = thr;
    m.csr_chunk = chunk;
    std::vector<int32_t> rp((size_t)m.R + 1);
    GS_HIP(hipMemcpyAsync(rp.data(), m.row_ptr.p, rp.size() * 4, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));

    // Skewed row lengths (coefficient of variation above 1/2): order by length.
    double sum = 0, sum2 = 0;
    for (int64_t i = 0; i < m.R; i++) {
        const double l = rp[i + 1] - rp[i];
        sum += l;
        sum2 += l * l;
    }
    const double mean = m.R ? sum / m.R : 0.0;
    const double var = m.R ? std::max(0.0, sum2 / m.R - mean * mean) : 0.0;
    const int force = env_int("GS_CSR_SORT", 0);  // 1: never, 2: always
    bool sorted = mean > 0 && std::sqrt(var) > 0.5 * mean;
    if (force == 1) sorted = false;
    if (force == 2) sorted = true;
    m.csr_sorted = sorted;

    std::vector<int32_t> lrows;
    std::vector<int4> shorts;
    shorts.reserve((size_t)m.R);
    for (int64_t i = 0; i < m.R; i++) {
        const int32_t a = rp[i], len = rp[i + 1] - rp[i];
        if (len > thr)
            lrows.push_back((int32_t)i);
        else
            shorts.push_back(make_int4((int)i, a, len, -1));
    }
    // medium long rows (one workgroup each on the vectorised path) first,
    // then huge ones (split across workgroups there); each in decreasing length
    const int wg_thr = env_int("GS_CSR_WG_ROW", kCsrWgRow);
    m.csr_wg_thr = wg_thr;
    std::stable_sort(lrows.begin(), lrows.end(), [&](int32_t p, int32_t q) {
        const int32_t lp = rp[p + 1] - rp[p], lq = rp[q + 1] - rp[q];
        const bool hp = lp > wg_thr, hq = lq > wg_thr;
        if (hp != hq) return hq;  // medium before huge
        return lp > lq;
    });
    m.n_medium_rows = 0;
    for (int32_t r : lrows) m.n_medium_rows += (rp[r + 1] - rp[r]) <= wg_thr;
    if (sorted) {  // stable counting sort by decreasing length (short rows have <= thr entries)
        std::vector<int64_t> start((size_t)thr + 2, 0);
        for (const int4 &it : shorts) start[(size_t)(thr - it.z) + 1]++;
        for (size_t i = 1; i < start.size(); i++) start[i] += start[i - 1];
        std::vector<int4> by_len(shorts.size());
        for (const int4 &it : shorts) by_len[(size_t)start[(size_t)(thr - it.z)]++] = it;
        shorts.swap(by_len);
    }
    std::vector<int4> items;
    std::vector<int32_t> lfirst;
    int32_t slot = 0;
    for (size_t k = 0; k < lrows.size(); k++) {
        const int32_t r = lrows[k];
        if ((int64_t)k == m.n_medium_rows) m.n_medium_chunks = slot;
        lfirst.push_back(slot);
        const int32_t a = rp[r], len = rp[r + 1] - rp[r];
        for (int32_t o = 0; o < len; o += chunk) items.push_back(make_int4(r, a + o, std::min(chunk, len - o), slot++));
    }
    if ((int64_t)lrows.size() == m.n_medium_rows) m.n_medium_chunks = slot;
    lfirst.push_back(slot);
    m.n_short = (int64_t)shorts.size();
    items.insert(items.end(), shorts.begin(), shorts.end());

    m.n_items = (int64_t)items.size();
    m.n_long_rows = (int64_t)lrows.size();
    m.n_long_chunks = slot;
    m.csr_items.alloc(items.size() * sizeof(int4), s);
    m.long_rows.alloc(lrows.size() * 4, s);
    m.long_first.alloc(lfirst.size() * 4, s);
    if (!items.empty())
        GS_HIP(hipMemcpyAsync(m.csr_items.p, items.data(), items.size() * sizeof(int4),
                              hipMemcpyHostToDevice, s));
    if (!lrows.empty())
        GS_HIP(hipMemcpyAsync(m.long_rows.p, lrows.data(), lrows.size() * 4, hipMemcpyHostToDevice, s));
    GS_HIP(hipMemcpyAsync(m.long_first.p, lfirst.data(), lfirst.size() * 4, hipMemcpyHostToDevice, s));
    GS_HIP(hipStreamSynchronize(s));
    m.csr_planned = true;
}

// ------------------------------------------------------------- launcher

bool spmm_csr_vec4(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                   hipStream_t s)
{
    auto al = [](const void *p) { return ((uintptr_t)p % 16) == 0; };
    if (F % 4 || ldx % 4 || ldy % 4 || !al(X) || !al(Y)) return false;
    // Lane shape: skewed (length-sorted) matrices gather rows at random, and
    // there wide groups (32 lanes, one X row per half-wave) do best; rows in
    // natural order do best with 16 columns per lane (more rows per wave).
    int cpl = env_int("GS_CSR_CPL", m.csr_sorted ? (int)std::max<int64_t>(4, std::min<int64_t>(16, F / 32)) : 16);
    if (cpl != 4 && cpl != 8 && cpl != 16) cpl = 16;
    while (cpl > 4 && F < 4 * (int64_t)cpl) cpl /= 2;  // at least 4 lanes per group
    const int64_t lanes = ceil_div(F, cpl);
    const int g = lanes <= 4 ? 4 : lanes <= 8 ? 8 : lanes <= 16 ? 16 : lanes <= 32 ? 32 : 64;
    const int64_t slices = ceil_div(F, (int64_t)g * cpl);
    const bool full = (F % ((int64_t)g * cpl)) == 0;
    auto launch = [&](auto cpl_t, auto g_t, auto full_t) {
        constexpr int CPL = decltype(cpl_t)::value, G = decltype(g_t)::value;
        constexpr bool FU = decltype(full_t)::value;
        constexpr int GPB = kBlock / G;
        const int64_t n_group_items = m.n_items - m.n_medium_chunks;  // huge chunks + short rows
        const int64_t n_huge = m.n_long_rows - m.n_medium_rows;
        const int64_t tiles = m.n_medium_rows + ceil_div(n_group_items, GPB);
        if (!tiles) return;
        if (n_huge) ensure_work(m, (size_t)m.n_long_chunks * F * 4, s);
        // persistent grid: a few resident workgroups per CU
        const int64_t cap = (int64_t)resident_workgroups() * env_int("GS_WG_MULT", 4);
        dim3 grid((unsigned)std::max<int64_t>(1, std::min(tiles, cap / slices)), (unsigned)slices);
        k_csr_rows<CPL, G, FU><<<grid, kBlock, 0, s>>>(
            m.n_medium_rows, m.long_rows.as<int32_t>(), m.row_ptr.as<int32_t>(), m.csr_chunk,
            n_group_items, m.csr_items.as<int4>() + m.n_medium_chunks, m.col.as<int32_t>(),
            m.val.as<float>(), X, ldx, Y, ldy, F, m.work.as<float>());
        GS_HIP(hipGetLastError());
        if (n_huge) {
            dim3 g2((unsigned)ceil_div(n_huge, GPB), (unsigned)slices);
            k_csr_combine<CPL, G><<<g2, kBlock, 0, s>>>(m.long_rows.as<int32_t>() + m.n_medium_rows,
                                                        m.long_first.as<int32_t>() + m.n_medium_rows,
                                                        n_huge, m.work.as<float>(), Y, ldy, F);
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
