// BSR SpMM with 16x16 blocks on the matrix cores (gfx950 MFMA).
//
// The default kernel is the hybrid one (k_bsr16_hybrid, further down): the
// handle's plan lists each block row's dense blocks (at least 64 of 256
// entries stored) for the matrix cores and keeps every other block's entries
// as rows gathered on the vector ALUs, so sparse blocks cost their entries.
// k_bsr16_mfma below runs every block from the block arrays alone.
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
#include <string>

#include "gs_device.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kBlock = 256;
// Blocks with at least this many of their 16 columns stored take the MFMA
// path; sparser ones are cheaper on the vector ALUs (an fp32 16x16x4 MFMA
// costs as much as 16 wave-wide FMAs per 4 block columns).
constexpr int kDenseCols = kBsrDenseCols;
// Blocks per running chain of an accumulator (16 products each).
constexpr int kFoldBlocks = kChainFold / 16;
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
        f32x4 acc[T], tot[T];
#pragma unroll
        for (int t = 0; t < T; t++) acc[t] = tot[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int64_t b0 = bptr[br], b1 = bptr[br + 1];
        // NB blocks per iteration: every load of the batch (masks, block
        // values, X rows) is issued before the first MFMA consumes one.
        for (int64_t blk = b0; blk < b1; blk += NB) {
            if (blk > b0 && (blk - b0) % kFoldBlocks == 0) {  // 16 terms per block into the running chain
#pragma unroll
                for (int t = 0; t < T; t++) {
                    tot[t] += acc[t];
                    acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
                }
            }
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
            tot[t] += acc[t];
            if (!tok[t]) continue;
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int64_t row = br * 16 + 4 * kk + i;
                if (row < R) __builtin_nontemporal_store(tot[t][i], Y + row * ldy + xcol + 16 * t);
            }
        }
    }
}

// Dense blocks on the matrix cores, the rest as a row list (hybrid plan).
//
// Wave w of a workgroup owns block row br = 4u + w and T consecutive
// 16-column tiles of F.  Phase 1 runs the block row's dense blocks (from the
// plan's list) on the matrix cores exactly as k_bsr16_mfma does.  Phase 2
// moves the 16 x 16T accumulator tile into the wave's own LDS rows and runs
// the block row's remaining entries (those of its sparse blocks, a CSR of
// their own) in the row layout of the CSR kernel: G = 4T lanes per row, a
// float4 of columns each, X rows gathered 8 at a time, the partial from
// phase 1 as the starting sum.  Y is written once.  A sparse block then
// costs its stored entries, not its 1 KiB of values and 16 X rows.
template <int T, int NB>
__global__ __launch_bounds__(kBlock) void k_bsr16_hybrid(
    int64_t R, int64_t nbr, const int32_t *__restrict__ dptr, const int32_t *__restrict__ didx,
    const int32_t *__restrict__ bcol, const float *__restrict__ bval, const uint64_t *__restrict__ bmask,
    const int32_t *__restrict__ rrp, const int32_t *__restrict__ rcol, const float *__restrict__ rval,
    const float *__restrict__ X, int64_t ldx, float *__restrict__ Y, int64_t ldy, int64_t F)
{
    constexpr int LDT = 16 * T + 4;  // floats per LDS row (padded: quadrants fall in other banks)
    constexpr int G = 4 * T;         // lanes per row in phase 2
    constexpr int P = kWave / G;     // rows per pass
    constexpr int U = G < 8 ? G : 8; // X rows in flight per batch
    __shared__ __align__(16) float tile[kBlock / kWave][16 * LDT];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int m = lane % 16, kk = lane / 16;
    const int64_t ntiles = F / 16;
    const int64_t tile0 = (int64_t)blockIdx.y * T;
    if (tile0 >= ntiles) return;  // whole workgroup idle (F narrower than the grid)
    bool tok[T];
#pragma unroll
    for (int t = 0; t < T; t++) tok[t] = tile0 + t < ntiles;
    const int64_t xcol = tile0 * 16 + m;
    float *tl = tile[wave];
    const int gl = lane % G, pr = lane / G;  // phase 2: lane in row group, row of the pass
    const bool cok = tok[gl / 4];            // phase 2: this lane's 4 columns lie inside F
    const int64_t c2 = tile0 * 16 + 4 * gl;
    const int64_t units = (nbr + 3) / 4;

    for (int64_t u = xcd_tile(blockIdx.x, gridDim.x); u < units; u += gridDim.x) {
        const int64_t br = u * 4 + wave;
        if (br >= nbr) break;
        f32x4 acc[T];
#pragma unroll
        for (int t = 0; t < T; t++) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        // every kFoldBlocks dense blocks (16 products each) the running sums
        // are added into the wave's LDS tile, which then holds the total
        bool folded = false;
        auto to_tile = [&](bool add) {
#pragma unroll
            for (int t = 0; t < T; t++)
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    float &c = tl[(4 * kk + i) * LDT + 16 * t + m];
                    c = add ? c + acc[t][i] : acc[t][i];
                }
        };
        const int64_t d0 = dptr[br], d1 = dptr[br + 1];
        for (int64_t d = d0; d < d1; d += NB) {
            if (d > d0 && (d - d0) % kFoldBlocks == 0) {
                to_tile(folded);
                folded = true;
#pragma unroll
                for (int t = 0; t < T; t++) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
            uint64_t mask[NB];
            int64_t xr0[NB];
            float av[NB][4];
#pragma unroll
            for (int j = 0; j < NB; j++) {
                const bool ok = d + j < d1;
                const int64_t blk = ok ? didx[d + j] : 0;
                mask[j] = ok ? bmask[blk] : 0ull;
                xr0[j] = ok ? (int64_t)bcol[blk] * 16 : 0;
                float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
                if (ok) a = *reinterpret_cast<const float4 *>(bval + blk * 256 + m * 16 + 4 * kk);
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
#pragma unroll
                    for (int t = 0; t < T; t++) bx[j][s][t] = (has && tok[t]) ? xp[16 * t] : 0.0f;
                }
#pragma unroll
            for (int j = 0; j < NB; j++)
#pragma unroll
                for (int s = 0; s < 4; s++) {
                    if (((mask[j] >> s) & 0x1111ull) == 0) continue;  // wave-uniform skip
#pragma unroll
                    for (int t = 0; t < T; t++)
                        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j][s], bx[j][s][t], acc[t], 0, 0, 0);
                }
        }
        // accumulator layout (lane m + 16 kk: rows 4kk..4kk+3, column m of
        // each tile) -> row-major tile in this wave's LDS rows
        to_tile(folded);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        for (int i0 = 0; i0 < 16; i0 += P) {
            const int i = i0 + pr;
            const int64_t row = br * 16 + i;
            float4 a = *reinterpret_cast<const float4 *>(tl + i * LDT + 4 * gl);
            if (row < R) {
                const int64_t k0 = rrp[row], k1 = rrp[row + 1];
                float4 run = make_float4(0.f, 0.f, 0.f, 0.f);  // the current chain of at most kChainFold terms
                for (int64_t kb = k0; kb < k1; kb += G) {
                    if (kb > k0 && (kb - k0) % kChainFold == 0) {
                        a.x += run.x;
                        a.y += run.y;
                        a.z += run.z;
                        a.w += run.w;
                        run = make_float4(0.f, 0.f, 0.f, 0.f);
                    }
                    const int mm = (k1 - kb) < G ? (int)(k1 - kb) : G;
                    int cj = 0;
                    float vj = 0.0f;
                    if (gl < mm) {
                        cj = ld_stream(rcol + kb + gl);
                        vj = ld_stream(rval + kb + gl);
                    }
                    for (int j = 0; j < mm; j += U) {
                        float4 x[U];
                        float v[U];
#pragma unroll
                        for (int e = 0; e < U; e++) {
                            const int cu = __shfl(cj, j + e, G);
                            v[e] = __shfl(vj, j + e, G);
                            x[e] = cok ? *reinterpret_cast<const float4 *>(X + (int64_t)cu * ldx + c2)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
                        }
#pragma unroll
                        for (int e = 0; e < U; e++) {
                            const bool live = j + e < mm;
                            const float a0 = __builtin_fmaf(v[e], x[e].x, run.x);
                            const float a1 = __builtin_fmaf(v[e], x[e].y, run.y);
                            const float a2 = __builtin_fmaf(v[e], x[e].z, run.z);
                            const float a3 = __builtin_fmaf(v[e], x[e].w, run.w);
                            run.x = live ? a0 : run.x;
                            run.y = live ? a1 : run.y;
                            run.z = live ? a2 : run.z;
                            run.w = live ? a3 : run.w;
                        }
                    }
                }
                a.x += run.x;
                a.y += run.y;
                a.z += run.z;
                a.w += run.w;
                if (cok) {
                    float *yp = Y + row * ldy + c2;
                    __builtin_nontemporal_store(a.x, yp);
                    __builtin_nontemporal_store(a.y, yp + 1);
                    __builtin_nontemporal_store(a.z, yp + 2);
                    __builtin_nontemporal_store(a.w, yp + 3);
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();  // the tile's LDS rows are rewritten by the next block row
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// ---- hybrid plan (built with a 16x16 BSR handle)

constexpr int kPB = 256;

inline unsigned pgrid(int64_t n)
{
    const int64_t g = (n + kPB - 1) / kPB;
    return (unsigned)(g < 1 ? 1 : g > 65535 ? 65535 : g);
}

// Entries per block: each row walks its entries and the blocks of its block
// row together (both in column order).
__global__ __launch_bounds__(kPB) void k_hyb_block_counts(const int32_t *__restrict__ rp,
                                                         const int32_t *__restrict__ col, int64_t R,
                                                         const int32_t *__restrict__ bptr,
                                                         const int32_t *__restrict__ bcol,
                                                         int32_t *__restrict__ cnt)
{
    for (int64_t r = (int64_t)blockIdx.x * kPB + threadIdx.x; r < R; r += (int64_t)gridDim.x * kPB) {
        int64_t p = bptr[r / 16];
        for (int64_t k = rp[r]; k < rp[r + 1]; k++) {
            const int c16 = col[k] / 16;
            while (bcol[p] < c16) p++;
            atomicAdd(&cnt[p], 1);
        }
    }
}

// Dense blocks (at least `dense_min` entries) per block row.
__global__ __launch_bounds__(kPB) void k_hyb_dense_rows(const int32_t *__restrict__ bptr, int64_t nbr,
                                                       const int32_t *__restrict__ cnt, int dense_min,
                                                       int32_t *__restrict__ dcnt)
{
    for (int64_t br = (int64_t)blockIdx.x * kPB + threadIdx.x; br < nbr; br += (int64_t)gridDim.x * kPB) {
        int n = 0;
        for (int64_t b = bptr[br]; b < bptr[br + 1]; b++) n += cnt[b] >= dense_min;
        dcnt[br] = n;
    }
}

__global__ __launch_bounds__(kPB) void k_hyb_dense_list(const int32_t *__restrict__ bptr, int64_t nbr,
                                                       const int32_t *__restrict__ cnt, int dense_min,
                                                       const int32_t *__restrict__ dptr,
                                                       int32_t *__restrict__ didx)
{
    for (int64_t br = (int64_t)blockIdx.x * kPB + threadIdx.x; br < nbr; br += (int64_t)gridDim.x * kPB) {
        int64_t o = dptr[br];
        for (int64_t b = bptr[br]; b < bptr[br + 1]; b++)
            if (cnt[b] >= dense_min) didx[o++] = (int32_t)b;
    }
}

// Entries of sparse blocks per row (WRITE = false: counts into rcnt; true:
// the entries into the remainder CSR at rrp[r]).
template <bool WRITE>
__global__ __launch_bounds__(kPB) void k_hyb_rest(const int32_t *__restrict__ rp, const int32_t *__restrict__ col,
                                                 const float *__restrict__ val, int64_t R,
                                                 const int32_t *__restrict__ bptr,
                                                 const int32_t *__restrict__ bcol,
                                                 const int32_t *__restrict__ cnt, int dense_min,
                                                 int32_t *__restrict__ rcnt, const int32_t *__restrict__ rrp,
                                                 int32_t *__restrict__ rcol, float *__restrict__ rval)
{
    for (int64_t r = (int64_t)blockIdx.x * kPB + threadIdx.x; r < R; r += (int64_t)gridDim.x * kPB) {
        int64_t p = bptr[r / 16];
        int64_t o = WRITE ? rrp[r] : 0;
        int n = 0;
        for (int64_t k = rp[r]; k < rp[r + 1]; k++) {
            const int c = col[k];
            while (bcol[p] < c / 16) p++;
            if (cnt[p] >= dense_min) continue;
            if (WRITE) {
                rcol[o] = c;
                rval[o] = val[k];
                o++;
            }
            n++;
        }
        if (!WRITE) rcnt[r] = n;
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

void plan_bsr_hybrid(gs_matrix_ &m, const int32_t *rp, const int32_t *col, const float *val, hipStream_t s)
{
    const char *e = std::getenv("GS_BSR_HYBRID");
    if ((e && std::string(e) == "off") || m.b != 16 || m.nb == 0) return;
    const int64_t R = m.R, nbr = ceil_div(R, 16);
    const int dense_min = env_int("GS_BSR_DENSE_MIN", kHybridDenseMin);
    DevBuf cnt, dcnt, rcnt;
    cnt.alloc((size_t)m.nb * 4, s);
    GS_HIP(hipMemsetAsync(cnt.p, 0, cnt.bytes, s));
    k_hyb_block_counts<<<pgrid(R), kPB, 0, s>>>(rp, col, R, m.bptr.as<int32_t>(), m.bcol.as<int32_t>(),
                                                cnt.as<int32_t>());
    GS_HIP(hipGetLastError());
    m.hyb_dptr.alloc((size_t)(nbr + 1) * 4, s);
    k_hyb_dense_rows<<<pgrid(nbr), kPB, 0, s>>>(m.bptr.as<int32_t>(), nbr, cnt.as<int32_t>(), dense_min,
                                                m.hyb_dptr.as<int32_t>());
    GS_HIP(hipGetLastError());
    exclusive_scan_i32(m.hyb_dptr.as<int32_t>(), m.hyb_dptr.as<int32_t>(), nbr, true, s);
    m.hyb_rrp.alloc((size_t)(R + 1) * 4, s);
    k_hyb_rest<false><<<pgrid(R), kPB, 0, s>>>(rp, col, val, R, m.bptr.as<int32_t>(), m.bcol.as<int32_t>(),
                                               cnt.as<int32_t>(), dense_min, m.hyb_rrp.as<int32_t>(), nullptr,
                                               nullptr, nullptr);
    GS_HIP(hipGetLastError());
    exclusive_scan_i32(m.hyb_rrp.as<int32_t>(), m.hyb_rrp.as<int32_t>(), R, true, s);
    int32_t tot[2] = {0, 0};
    GS_HIP(hipMemcpyAsync(&tot[0], m.hyb_dptr.as<int32_t>() + nbr, 4, hipMemcpyDeviceToHost, s));
    GS_HIP(hipMemcpyAsync(&tot[1], m.hyb_rrp.as<int32_t>() + R, 4, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));
    m.hyb_ndense = tot[0];
    m.hyb_nrest = tot[1];
    m.hyb_didx.alloc((size_t)m.hyb_ndense * 4, s);
    m.hyb_rcol.alloc((size_t)m.hyb_nrest * 4, s);
    m.hyb_rval.alloc((size_t)m.hyb_nrest * 4, s);
    if (m.hyb_ndense) {
        k_hyb_dense_list<<<pgrid(nbr), kPB, 0, s>>>(m.bptr.as<int32_t>(), nbr, cnt.as<int32_t>(), dense_min,
                                                    m.hyb_dptr.as<int32_t>(), m.hyb_didx.as<int32_t>());
        GS_HIP(hipGetLastError());
    }
    if (m.hyb_nrest) {
        k_hyb_rest<true><<<pgrid(R), kPB, 0, s>>>(rp, col, val, R, m.bptr.as<int32_t>(), m.bcol.as<int32_t>(),
                                                  cnt.as<int32_t>(), dense_min, nullptr, m.hyb_rrp.as<int32_t>(),
                                                  m.hyb_rcol.as<int32_t>(), m.hyb_rval.as<float>());
        GS_HIP(hipGetLastError());
    }
    m.hyb_planned = true;
}

// The hybrid kernel: F a multiple of 16, X / Y 16-byte aligned rows.
bool spmm_bsr16_hybrid(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                       hipStream_t s)
{
    auto al = [](const void *p) { return ((uintptr_t)p % 16) == 0; };
    if (!m.hyb_planned || F % 16 || ldx % 4 || ldy % 4 || !al(X) || !al(Y)) return false;
    if (env_int("GS_BSR_GENERIC", 0) || env_int("GS_BSR_MFMA", 0)) return false;
    const int64_t nbr = ceil_div(m.R, 16);
    if (nbr == 0) return true;
    const int64_t ntiles = F / 16;
    // 4 tiles (64 columns) per wave and about 8 workgroups per CU: on the
    // block-community graph (F = 256) 2 / 4 / 8 tiles measured 259 / 211 /
    // 289 us (8 tiles hold 153 VGPRs: 2 waves per SIMD), the mesh 55 / 57 /
    // 130 us.
    int T = ntiles <= 1 ? 1 : ntiles <= 2 ? 2 : 4;
    if (const int ht = env_int("GS_BSR_HT", 0); ht == 1 || ht == 2 || ht == 4 || ht == 8) T = ht;  // sweeps
    const int64_t ygroups = ceil_div(ntiles, T), units = ceil_div(nbr, 4);
    const int64_t cap = (int64_t)resident_workgroups() * env_int("GS_WG_MULT", 8);
    dim3 grid((unsigned)std::max<int64_t>(1, std::min(units, cap / ygroups)), (unsigned)ygroups);
#define GS_H(TT)                                                                                            \
    k_bsr16_hybrid<TT, 2><<<grid, kBlock, 0, s>>>(m.R, nbr, m.hyb_dptr.as<int32_t>(), m.hyb_didx.as<int32_t>(), \
                                                  m.bcol.as<int32_t>(), m.bval.as<float>(),                     \
                                                  m.bmask.as<uint64_t>(), m.hyb_rrp.as<int32_t>(),              \
                                                  m.hyb_rcol.as<int32_t>(), m.hyb_rval.as<float>(), X, ldx, Y,  \
                                                  ldy, F)
    switch (T) {
    case 1: GS_H(1); break;
    case 2: GS_H(2); break;
    case 4: GS_H(4); break;
    default: GS_H(8); break;
    }
#undef GS_H
    GS_HIP(hipGetLastError());
    return true;
}

bool spmm_bsr16_mfma(gs_matrix_ &m, const float *X, int64_t ldx, float *Y, int64_t ldy, int64_t F,
                     hipStream_t s)
{
    if (spmm_bsr16_hybrid(m, X, ldx, Y, ldy, F, s)) return true;
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
