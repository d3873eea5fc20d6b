// CSR SpMM, vectorised path (F a multiple of 4, 16-byte aligned operands).
//
// The matrix is cut at plan time into work items {row, start, len, slot}:
// one item per row of at most `long_thr` entries, and chunks of `chunk`
// entries for longer rows (slot >= 0: the chunk's partial sum goes to
// work[slot*F...] and a second launch adds a long row's chunks in order).
// For rows with skewed lengths (power-law graphs) the items are ordered by
// decreasing length, so the rows sharing a wavefront have equal trip counts
// and the longest work starts first; otherwise rows keep their natural
// order (neighbouring rows share X rows in L2).
//
// A group of G lanes owns one item; lane l holds CPL consecutive columns
// (CPL/4 float4 per X row), so a group covers G*CPL columns and a wave
// holds 64/G items.  Entries are fetched G at a time (one per lane) and
// broadcast by shuffles; X rows are then gathered U at a time (U*CPL/4 =
// 8 float4 loads in flight per lane) before any of them is consumed.  The
// last batch of a row is masked (a select, so Inf/NaN in X cannot leak in
// through a masked slot).
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

template <int CPL, int G, bool FULL, int LIF>
__global__ __launch_bounds__(kBlock) void k_csr_items(int64_t n_items, const int4 *__restrict__ items,
                                                      const int32_t *__restrict__ col,
                                                      const float *__restrict__ val,
                                                      const float *__restrict__ X, int64_t ldx,
                                                      float *__restrict__ Y, int64_t ldy, int64_t F,
                                                      float *__restrict__ work, int xs)
{
    constexpr int GPB = kBlock / G;
    constexpr int NQ = CPL / 4;
    constexpr int U0 = (4 * LIF / CPL) > 0 ? 4 * LIF / CPL : 1;  // LIF float4 loads in flight per lane
    constexpr int U = U0 < G ? U0 : G;  // never more than one index batch
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    // Column slice and first row tile of this workgroup.  With xs > 0 the
    // slices are pinned to XCDs (workgroup ids reach the 8 XCDs
    // round-robin): XCD x serves slice x % xs only, so its L2 caches 1/xs of
    // every X row.  The grid is persistent: each workgroup walks row tiles
    // with a stride of the number of workgroups serving its slice.
    int64_t tile, tstride;
    int slice;
    if (xs > 0) {
        const int x = (int)(blockIdx.x % kXcds);
        tile = (int64_t)(blockIdx.x / kXcds) * (kXcds / xs) + x / xs;
        tstride = (int64_t)(gridDim.x / kXcds) * (kXcds / xs);
        slice = x % xs;
    } else {
        tile = blockIdx.x;
        tstride = gridDim.x;
        slice = blockIdx.y;
    }
    // float4 q of this lane sits at column base + (q*G + lane)*4, so one
    // load instruction covers G*16 contiguous bytes of an X row.
    const int64_t c0 = (int64_t)slice * (G * CPL) + (int64_t)lane * 4;
    bool qok[NQ];
#pragma unroll
    for (int q = 0; q < NQ; q++) qok[q] = FULL || (c0 + 4 * G * q < F);

    for (; tile * GPB < n_items; tile += tstride) {
    const int64_t it = tile * GPB + g;
    if (it >= n_items) break;
    const int4 d = items[it];
    float acc[CPL];
#pragma unroll
    for (int i = 0; i < CPL; i++) acc[i] = 0.0f;

    int64_t kb = d.y;
    int rem = d.z;
    while (rem > 0) {
        const int m = rem < G ? rem : G;
        int cj = 0;
        float vj = 0.0f;
        if (lane < m) {
            cj = ld_stream(col + kb + lane);
            vj = ld_stream(val + kb + lane);
        }
        int j = 0;
        for (; j + U <= m; j += U) gather_batch<U, NQ, G, false>(cj, vj, j, m, X, ldx, c0, qok, acc);
        // tail: a masked batch of U/2 or U entries, whichever covers it
        if (j < m) {
            if (U > 1 && m - j <= U / 2)
                gather_batch<(U > 1 ? U / 2 : 1), NQ, G, true>(cj, vj, j, m, X, ldx, c0, qok, acc);
            else
                gather_batch<U, NQ, G, true>(cj, vj, j, m, X, ldx, c0, qok, acc);
        }
        kb += m;
        rem -= m;
    }
    if (d.w < 0) {
        float *yp = Y + (int64_t)d.x * ldy + c0;
#pragma unroll
        for (int q = 0; q < NQ; q++)
            if (qok[q]) {
#pragma unroll
                for (int i = 0; i < 4; i++) __builtin_nontemporal_store(acc[4 * q + i], yp + 4 * G * q + i);
            }
    } else {
        float *wp = work + (int64_t)d.w * F + c0;
#pragma unroll
        for (int q = 0; q < NQ; q++)
            if (qok[q])
                *reinterpret_cast<float4 *>(wp + 4 * G * q) =
                    make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
    }
    }  // tile loop
}

// One group per long row: adds its chunks' partials (consecutive slots) in
// slot order and writes the row of Y.
template <int CPL, int G>
__global__ __launch_bounds__(kBlock) void k_csr_combine4(const int32_t *__restrict__ long_rows,
                                                         const int32_t *__restrict__ long_first,
                                                         int64_t n_long, const float *__restrict__ work,
                                                         float *__restrict__ Y, int64_t ldy, int64_t F)
{
    constexpr int GPB = kBlock / G;
    constexpr int NQ = CPL / 4;
    const int g = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t lr = (int64_t)blockIdx.x * GPB + g;
    if (lr >= n_long) return;
    const int64_t c0 = (int64_t)blockIdx.y * (G * CPL) + (int64_t)lane * CPL;
    const int64_t s0 = long_first[lr], s1 = long_first[lr + 1];
    for (int q = 0; q < NQ; q++) {
        if (c0 + 4 * q >= F) break;
        const float *wp = work + c0 + 4 * q;
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
        int64_t sl = s0;
        // eight partials in flight; added strictly in slot order
        for (; sl + 8 <= s1; sl += 8) {
            float4 p[8];
#pragma unroll
            for (int u = 0; u < 8; u++) p[u] = *reinterpret_cast<const float4 *>(wp + (sl + u) * F);
#pragma unroll
            for (int u = 0; u < 8; u++) {
                a.x += p[u].x;
                a.y += p[u].y;
                a.z += p[u].z;
                a.w += p[u].w;
            }
        }
        for (; sl < s1; sl++) {
            const float4 p = *reinterpret_cast<const float4 *>(wp + sl * F);
            a.x += p.x;
            a.y += p.y;
            a.z += p.z;
            a.w += p.w;
        }
        float *yp = Y + (int64_t)long_rows[lr] * ldy + c0 + 4 * q;
        __builtin_nontemporal_store(a.x, yp + 0);
        __builtin_nontemporal_store(a.y, yp + 1);
        __builtin_nontemporal_store(a.z, yp + 2);
        __builtin_nontemporal_store(a.w, yp + 3);
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

    std::vector<int4> items;
    items.reserve((size_t)m.R + 16);
    std::vector<int32_t> lrows, lfirst;
    int32_t slot = 0;
    for (int64_t i = 0; i < m.R; i++) {
        const int32_t a = rp[i], len = rp[i + 1] - rp[i];
        if (len <= thr) continue;
        lrows.push_back((int32_t)i);
        lfirst.push_back(slot);
        for (int32_t o = 0; o < len; o += chunk)
            items.push_back(make_int4((int)i, a + o, std::min(chunk, len - o), slot++));
    }
    lfirst.push_back(slot);
    for (int64_t i = 0; i < m.R; i++) {
        const int32_t a = rp[i], len = rp[i + 1] - rp[i];
        if (len <= thr) items.push_back(make_int4((int)i, a, len, -1));
    }
    if (sorted)
        std::stable_sort(items.begin(), items.end(),
                         [](const int4 &p, const int4 &q) { return p.z > q.z; });

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
}

// ------------------------------------------------------------- launcher

bool spmm_csr_vec4(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                   hipStream_t s)
{
    auto al = [](const void *p) { return ((uintptr_t)p % 16) == 0; };
    if (F % 4 || ldx % 4 || ldy % 4 || !al(X) || !al(Y)) return false;
    if (m.n_long_chunks) ensure_work(m, (size_t)m.n_long_chunks * F * 4, s);
    // XCD slicing: xs column slices of F, each pinned to 8/xs XCDs.
    int xs = env_int("GS_CSR_XSLICE", 1);
    if (xs != 1 && xs != 2 && xs != 4 && xs != 8) xs = 1;
    int cpl, g;
    int64_t slices;
    bool full;
    // Lane shape: skewed (length-sorted) matrices gather rows at random, and
    // there wide groups (32 lanes, one X row per half-wave) do best; rows in
    // natural order do best with 16 columns per lane (more rows per wave).
    const int want_cpl = env_int("GS_CSR_CPL", m.csr_sorted ? (F >= 128 ? (int)std::max<int64_t>(4, F / 32) : 4) : 16);
    const int lif = env_int("GS_CSR_LIF", 8) >= 16 ? 16 : 8;
    if (F % (4 * xs) == 0 && F / xs <= 1024 && (F / xs) % 16 == 0) {
        const int64_t w = F / xs;  // columns per slice
        cpl = w >= 8 * want_cpl ? want_cpl : (w >= 64 ? 8 : 4);
        g = (int)(w / cpl);
        if (g > 64) { g = 64; cpl = (int)(w / 64); }
        if (cpl != 4 && cpl != 8 && cpl != 16) { cpl = 4; g = (int)(w / 4); }
        slices = xs;
        full = true;
    } else {
        xs = 0;
        cpl = (F % 8 == 0) ? 8 : 4;
        int64_t lanes = ceil_div(F, cpl);
        g = lanes <= 8 ? 8 : lanes <= 16 ? 16 : lanes <= 32 ? 32 : 64;
        slices = ceil_div(F, (int64_t)g * cpl);
        full = (F % ((int64_t)g * cpl)) == 0;
    }
    const int4 *items = m.csr_items.as<int4>();
    auto launch = [&](auto cpl_t, auto g_t, auto full_t, auto lif_t) {
        constexpr int CPL = decltype(cpl_t)::value, G = decltype(g_t)::value;
        constexpr bool FU = decltype(full_t)::value;
        constexpr int LIF = decltype(lif_t)::value;
        constexpr int GPB = kBlock / G;
        if (m.n_items) {
            const int64_t tiles = ceil_div(m.n_items, GPB);
            // persistent grid: enough workgroups to fill every CU, no more
            const int64_t cap = (int64_t)resident_workgroups() * env_int("GS_WG_MULT", 4);
            dim3 grid;
            if (xs > 0) {
                int64_t per_slice = std::min(ceil_div(tiles, kXcds / xs), ceil_div(cap, kXcds));
                grid = dim3((unsigned)(per_slice * kXcds), 1);
            } else {
                grid = dim3((unsigned)std::min(tiles, std::max<int64_t>(1, cap / slices)), (unsigned)slices);
            }
            k_csr_items<CPL, G, FU, LIF><<<grid, kBlock, 0, s>>>(m.n_items, items, m.col.as<int32_t>(),
                                                            m.val.as<float>(), X, ldx, Y, ldy, F,
                                                            m.work.as<float>(), xs);
            GS_HIP(hipGetLastError());
        }
        if (m.n_long_rows) {
            dim3 g2((unsigned)ceil_div(m.n_long_rows, GPB), (unsigned)slices);
            k_csr_combine4<CPL, G><<<g2, kBlock, 0, s>>>(m.long_rows.as<int32_t>(),
                                                         m.long_first.as<int32_t>(), m.n_long_rows,
                                                         m.work.as<float>(), Y, ldy, F);
            GS_HIP(hipGetLastError());
        }
    };
    using I = std::integral_constant<int, 0>;
    (void)sizeof(I);
#define GS_L(C, GG)                                                                       \
    if (cpl == C && g == GG) {                                                            \
        using CI = std::integral_constant<int, C>;                                        \
        using GI = std::integral_constant<int, GG>;                                       \
        using L8 = std::integral_constant<int, 8>;                                        \
        using L16 = std::integral_constant<int, 16>;                                      \
        if (full && lif == 16) launch(CI{}, GI{}, std::true_type{}, L16{});               \
        else if (full) launch(CI{}, GI{}, std::true_type{}, L8{});                        \
        else launch(CI{}, GI{}, std::false_type{}, L8{});                                 \
        return true;                                                                      \
    }
    GS_L(16, 4) GS_L(16, 8) GS_L(16, 16) GS_L(16, 32) GS_L(16, 64)
    GS_L(8, 8) GS_L(8, 16) GS_L(8, 32) GS_L(8, 64)
    GS_L(4, 4) GS_L(4, 8) GS_L(4, 16) GS_L(4, 32) GS_L(4, 64)
#undef GS_L
    return false;
}

}  // namespace gs
