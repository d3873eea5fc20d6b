// BSR SpMM with 16x16 blocks on the matrix cores (gfx950 MFMA).
//
// A 16x16 block B times the 16 X rows of its block column is a dense
// 16x16x16 contraction per 16-column tile of F.  It is issued as four
// V_MFMA_F32_16X16X4_F32 steps: step s takes block columns {s, 4+s, 8+s,
// 12+s}, so that lane l (m = l%16, kk = l/16) holds B[m][4kk .. 4kk+3] for all
// four steps after ONE coalesced float4 load of the block (the whole 1 KiB
// block per wave instruction, straight into the A operands; nothing is
// staged in LDS because nothing is reused across waves).  The B operand of
// step s is X[bc*16 + 4kk + s][tile*16 + m]: lanes gather X rows only for
// block columns that hold a nonzero (the block's column mask), and a step
// whose four columns are all empty is skipped entirely, so a sparse block
// costs its 1 KiB of values plus its touched X rows, and a full block is a
// true dense contraction.
//
// Workgroup = 4 waves on one block row; wave w owns T consecutive 16-column
// tiles of F (grid.y covers wider F), accumulating its 16 x 16T output tile
// in MFMA accumulator layout (lane l holds rows 4kk..4kk+3 of column m).  The
// grid is persistent over block rows in natural order (XCD-contiguous), so
// block rows of one community share X rows in one L2.
#include <algorithm>
#include <cstdlib>

#include "gs_device.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kBlock = 256;
// Blocks with at least this many of their 16 columns stored take the MFMA
// path; sparser ones are cheaper on the vector ALUs (an fp32 16x16x4 MFMA
// costs as much as 16 wave-wide FMAs per 4 block columns).
constexpr int kDenseCols = kBsrDenseCols;
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int T, int NB, bool WROWS>
__global__ __launch_bounds__(kBlock) void k_bsr16_mfma(int64_t R, int64_t nbr,
                                                       const int32_t *__restrict__ bptr,
                                                       const int32_t *__restrict__ bcol,
                                                       const float *__restrict__ bval,
                                                       const uint64_t *__restrict__ bmask,
                                                       const float *__restrict__ X, int64_t ldx,
                                                       float *__restrict__ Y, int64_t ldy, int64_t F)
{
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int m = lane % 16, kk = lane / 16;
    const int64_t ntiles = F / 16;
    // WROWS: the 4 waves own 4 different block rows and share one group of T
    // tiles (per-block work paid once per tile group); otherwise the 4 waves
    // share one block row and split 4*T tiles.
    const int64_t tile0 = WROWS ? (int64_t)blockIdx.y * T : ((int64_t)blockIdx.y * 4 + wave) * T;
    if (tile0 >= ntiles) return;  // whole wave idle (F narrower than the grid)
    bool tok[T];
#pragma unroll
    for (int t = 0; t < T; t++) tok[t] = tile0 + t < ntiles;
    const int64_t xcol = tile0 * 16 + m;
    const int64_t units = WROWS ? (nbr + 3) / 4 : nbr;

    for (int64_t u = xcd_tile(blockIdx.x, gridDim.x); u < units; u += gridDim.x) {
        const int64_t br = WROWS ? u * 4 + wave : u;
        if (br >= nbr) break;
        f32x4 acc[T];
#pragma unroll
        for (int t = 0; t < T; t++) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int64_t b0 = bptr[br], b1 = bptr[br + 1];
        // NB blocks per iteration: every load of the batch (masks, block
        // values, X rows) is issued before the first MFMA consumes one.
        for (int64_t blk = b0; blk < b1; blk += NB) {
            uint64_t mask[NB];
            int64_t xr0[NB];
            float av[NB][4];
#pragma unroll
            for (int j = 0; j < NB; j++) {
                const bool ok = blk + j < b1;
                mask[j] = ok ? bmask[blk + j] : 0ull;
                xr0[j] = ok ? (int64_t)bcol[blk + j] * 16 : 0;
            }
#pragma unroll
            for (int j = 0; j < NB; j++) {
                float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
                if (mask[j]) a = *reinterpret_cast<const float4 *>(bval + (blk + j) * 256 + m * 16 + 4 * kk);
                av[j][0] = a.x;
                av[j][1] = a.y;
                av[j][2] = a.z;
                av[j][3] = a.w;
            }
            float bx[NB][4][T];
#pragma unroll
            for (int j = 0; j < NB; j++)
#pragma unroll
                for (int s = 0; s < 4; s++) {
                    const int c = 4 * kk + s;
                    const bool has = (mask[j] >> c) & 1ull;
                    const float *xp = X + (xr0[j] + c) * ldx + xcol;
                    if (((mask[j] >> s) & 0x1111ull) == 0) {  // wave-uniform: no load issued
#pragma unroll
                        for (int t = 0; t < T; t++) bx[j][s][t] = 0.0f;
                        continue;
                    }
#pragma unroll
                    for (int t = 0; t < T; t++) bx[j][s][t] = (has && tok[t]) ? xp[16 * t] : 0.0f;
                }
#pragma unroll
            for (int j = 0; j < NB; j++) {
                if (__popcll(mask[j]) >= kDenseCols) {
                    // dense enough: the block times its X tile on the matrix cores
#pragma unroll
                    for (int s = 0; s < 4; s++) {
                        if (((mask[j] >> s) & 0x1111ull) == 0) continue;  // wave-uniform skip
#pragma unroll
                        for (int t = 0; t < T; t++)
                            acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j][s], bx[j][s][t], acc[t], 0, 0, 0);
                    }
                } else {
                    // sparse block: per stored column c, the 16 values B[.][c] and
                    // the gathered X row are broadcast to the accumulator layout
                    // (lane m + 16*kk owns rows 4kk..4kk+3 of column m) by shuffles
#pragma unroll
                    for (int s = 0; s < 4; s++)
#pragma unroll
                        for (int q = 0; q < 4; q++) {
                            if (!((mask[j] >> (4 * q + s)) & 1ull)) continue;  // wave-uniform
                            const int src = 16 * q;  // lanes holding block column 4q+s
                            float bvs[4];
#pragma unroll
                            for (int i = 0; i < 4; i++) bvs[i] = __shfl(av[j][s], 4 * kk + i + src, kWave);
#pragma unroll
                            for (int t = 0; t < T; t++) {
                                const float xv = __shfl(bx[j][s][t], m + src, kWave);
#pragma unroll
                                for (int i = 0; i < 4; i++) acc[t][i] = __builtin_fmaf(bvs[i], xv, acc[t][i]);
                            }
                        }
                }
            }
        }
#pragma unroll
        for (int t = 0; t < T; t++) {
            if (!tok[t]) continue;
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int64_t row = br * 16 + 4 * kk + i;
                if (row < R) __builtin_nontemporal_store(acc[t][i], Y + row * ldy + xcol + 16 * t);
            }
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

bool spmm_bsr16_mfma(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                     hipStream_t s)
{
    if (m.b != 16 || F % 16 != 0 || env_int("GS_BSR_GENERIC", 0)) return false;
    // Measured crossover: with few dense blocks the per-block overhead of the
    // matrix-core kernel loses to the generic column-skipping kernel.
    if (m.nb > 0 && m.n_dense_blocks * 10 < m.nb && !env_int("GS_BSR_MFMA", 0)) return false;
    const int64_t nbr = ceil_div(m.R, 16);
    if (nbr == 0) return true;
    const int64_t ntiles = F / 16;
    // tiles per wave: a workgroup's 4 waves cover 4*T tiles; wider F uses grid.y
    const bool wrows = env_int("GS_BSR_WROWS", 2) == 1;  // 1: one block row per wave
    int T;
    int64_t ygroups, units;
    if (wrows) {
        T = ntiles <= 1 ? 1 : ntiles <= 2 ? 2 : ntiles <= 4 ? 4 : 8;
        ygroups = ceil_div(ntiles, T);
        units = ceil_div(nbr, 4);
    } else {
        T = ntiles <= 4 ? 1 : ntiles <= 8 ? 2 : ntiles <= 16 ? 4 : 8;
        ygroups = ceil_div(ntiles, 4 * T);
        units = nbr;
    }
    const int64_t cap = (int64_t)resident_workgroups() * env_int("GS_WG_MULT", 2);
    const unsigned gx = (unsigned)std::max<int64_t>(1, std::min(units, cap / ygroups));
    dim3 grid(gx, (unsigned)ygroups);
    const int32_t *bp = m.bptr.as<int32_t>(), *bc = m.bcol.as<int32_t>();
    const float *bv = m.bval.as<float>();
    const uint64_t *bm = m.bmask.as<uint64_t>();
    const int nb = env_int("GS_BSR_NB", 2) >= 4 ? 4 : 2;
#define GS_B(TT, NN, WW) \
    k_bsr16_mfma<TT, NN, WW><<<grid, kBlock, 0, s>>>(m.R, nbr, bp, bc, bv, bm, X, ldx, Y, ldy, F)
#define GS_T(NN, WW)                     \
    switch (T) {                         \
    case 1: GS_B(1, NN, WW); break;      \
    case 2: GS_B(2, NN, WW); break;      \
    case 4: GS_B(4, NN, WW); break;      \
    default: GS_B(8, 2, WW); break;      \
    }
    if (wrows) {
        if (nb == 4) { GS_T(4, true) } else { GS_T(2, true) }
    } else {
        if (nb == 4) { GS_T(4, false) } else { GS_T(2, false) }
    }
#undef GS_T
#undef GS_B
    GS_HIP(hipGetLastError());
    return true;
}

}  // namespace gs
