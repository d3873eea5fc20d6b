// Matrix features of the format predictor (Sec. 4.4, Table 2), extracted on
// the device from the canonical CSR form.  The device produces integer
// aggregates only (row/column counts and their max, min, sum of squares and
// sum of adjacent absolute differences; the number of occupied diagonals;
// the number of occupied 16x16 blocks), combined with integer atomics, so
// the result is exact and deterministic.  The 19 doubles are then formed on
// the host from those integers in one fixed operation order.
#include <climits>
#include <cmath>

#include "gs_device.h"
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

// Statistics of a count sequence cnt[i] = (ptr ? ptr[i+1]-ptr[i] : vals[i]).
__global__ __launch_bounds__(kTB) void k_count_stats(const int32_t *__restrict__ ptr,
                                                     const int32_t *__restrict__ vals, int64_t n,
                                                     int is_row, FeatAcc *__restrict__ acc)
{
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
    s2 = wave_sum_u64(s2);
    bn = wave_sum_u64(bn);
    mx = wave_max_i32(mx);
    mn = wave_min_i32(mn);
    if (lane_id() == 0) {
        if (is_row) {
            atomicAdd(&acc->s2r, s2);
            atomicAdd(&acc->bnr, bn);
            atomicMax(&acc->maxr, mx);
            atomicMin(&acc->minr, mn);
        } else {
            atomicAdd(&acc->s2c, s2);
            atomicAdd(&acc->bnc, bn);
            atomicMax(&acc->maxc, mx);
            atomicMin(&acc->minc, mn);
        }
    }
}

// One wavefront per row: lanes stride over the row's entries and mark the
// diagonal (col - row) each one lies on.
__global__ __launch_bounds__(kTB) void k_mark_diags(const int32_t *__restrict__ rp,
                                                    const int32_t *__restrict__ col, int64_t R,
                                                    uint32_t *__restrict__ bm)
{
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kTB / kWave);
    for (int64_t i = ((int64_t)blockIdx.x * kTB + threadIdx.x) / kWave; i < R; i += waves) {
        for (int64_t k = rp[i] + lane; k < rp[i + 1]; k += kWave) {
            int64_t sidx = (int64_t)col[k] - i + R - 1;
            // bits only ever get set: skip the atomic when the word already has it
            // (the main diagonal alone gets one hit per row)
            const uint32_t bit = 1u << (sidx & 31);
            if (!(__hip_atomic_load(&bm[sidx >> 5], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & bit))
                atomicOr(&bm[sidx >> 5], bit);
        }
    }
}

__global__ __launch_bounds__(kTB) void k_popc_total(const uint32_t *__restrict__ bm, int64_t nw,
                                                    unsigned long long *__restrict__ total)
{
    unsigned long long s = 0;
    for (int64_t w = (int64_t)blockIdx.x * kTB + threadIdx.x; w < nw;
         w += (int64_t)gridDim.x * kTB)
        s += __popc(bm[w]);
    s = wave_sum_u64(s);
    if (lane_id() == 0 && s) atomicAdd(total, s);
}

// R*S2 - Z^2 >= 0 (Cauchy-Schwarz), formed exactly in 128-bit arithmetic.
double population_dev(int64_t n, int64_t Z, uint64_t s2)
{
    if (n <= 0) return 0.0;
    unsigned __int128 num = (unsigned __int128)(uint64_t)n * s2 -
                            (unsigned __int128)(uint64_t)Z * (uint64_t)Z;
    double q = (double)num / ((double)n * (double)n);
    return std::sqrt(q);
}

}  // namespace

void features_from_csr(const gs_matrix_ &csr, hipStream_t s, gs_features *out)
{
    const int64_t R = csr.R, C = csr.C, Z = csr.Z;
    const int32_t *rp = csr.row_ptr.as<int32_t>();
    const int32_t *col = csr.col.as<int32_t>();

    FeatAcc h = {0, 0, 0, 0, 0, INT_MAX, 0, INT_MAX};
    unsigned long long nd = 0;
    DevBuf acc, cc, bm, ndv;
    acc.alloc(sizeof(FeatAcc), s);
    ndv.alloc(sizeof(unsigned long long), s);
    GS_HIP(hipMemcpyAsync(acc.p, &h, sizeof h, hipMemcpyHostToDevice, s));
    GS_HIP(hipMemsetAsync(ndv.p, 0, sizeof(unsigned long long), s));
    if (R > 0) {
        k_count_stats<<<elem_grid(R), kTB, 0, s>>>(rp, nullptr, R, 1, acc.as<FeatAcc>());
        GS_HIP(hipGetLastError());
    }
    if (C > 0) {
        cc.alloc((size_t)C * 4, s);
        GS_HIP(hipMemsetAsync(cc.p, 0, (size_t)C * 4, s));
        if (Z > 0) {
            k_col_hist<<<elem_grid(Z), kTB, 0, s>>>(col, Z, cc.as<int32_t>());
            GS_HIP(hipGetLastError());
        }
        k_count_stats<<<elem_grid(C), kTB, 0, s>>>(nullptr, cc.as<int32_t>(), C, 0, acc.as<FeatAcc>());
        GS_HIP(hipGetLastError());
    }
    if (Z > 0) {
        const int64_t nw = ceil_div(R + C - 1, 32);
        bm.alloc((size_t)nw * 4, s);
        GS_HIP(hipMemsetAsync(bm.p, 0, (size_t)nw * 4, s));
        k_mark_diags<<<elem_grid(R * kWave), kTB, 0, s>>>(rp, col, R, bm.as<uint32_t>());
        GS_HIP(hipGetLastError());
        k_popc_total<<<elem_grid(nw), kTB, 0, s>>>(bm.as<uint32_t>(), nw, ndv.as<unsigned long long>());
        GS_HIP(hipGetLastError());
    }
    GS_HIP(hipMemcpyAsync(&h, acc.p, sizeof h, hipMemcpyDeviceToHost, s));
    GS_HIP(hipMemcpyAsync(&nd, ndv.p, sizeof nd, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));
    const int64_t nb16 = count_blocks(csr, 16, s);

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

    const double dR = (double)R, dC = (double)C, dZ = (double)Z;
    const double aver_rd = R > 0 ? dZ / dR : 0.0;
    const double aver_cd = C > 0 ? dZ / dC : 0.0;
    const double dev_rd = population_dev(R, Z, f.sum_rd2);
    const double dev_cd = population_dev(C, Z, f.sum_cd2);
    double *F = f.f;
    F[0] = dR;                         // F1  numRow
    F[1] = dC;                         // F2  numCol
    F[2] = dZ;                         // F3  NNZ
    F[3] = (double)f.n_diags;          // F4  N_diags
    F[4] = aver_rd;                    // F5  aver_RD
    F[5] = (double)f.max_rd;           // F6  max_RD
    F[6] = (double)f.min_rd;           // F7  min_RD
    F[7] = dev_rd;                     // F8  dev_RD
    F[8] = aver_cd;                    // F9  aver_CD
    F[9] = (double)f.max_cd;           // F10 max_CD
    F[10] = (double)f.min_cd;          // F11 min_CD
    F[11] = dev_cd;                    // F12 dev_CD
    F[12] = (f.n_diags > 0 && R > 0) ? dZ / ((double)f.n_diags * dR) : 0.0;  // F13 ER_DIA
    F[13] = (C > 0 && f.max_cd > 0) ? dZ / (dC * (double)f.max_cd) : 0.0;    // F14 ER_CD
    F[14] = R > 1 ? (double)f.bounce_r / (double)(R - 1) : 0.0;              // F15 row_bounce
    F[15] = C > 1 ? (double)f.bounce_c / (double)(C - 1) : 0.0;              // F16 col_bounce
    F[16] = (R > 0 && C > 0) ? dZ / (dR * dC) : 0.0;                         // F17 density
    F[17] = aver_rd != 0.0 ? dev_rd / aver_rd : 0.0;                         // F18 cv
    F[18] = (double)f.max_rd - aver_rd;                                      // F19 max_mu
}

}  // namespace gs
