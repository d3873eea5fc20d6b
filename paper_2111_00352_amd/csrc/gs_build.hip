// Format construction on the device: validation and canonical ordering of
// the input COO, CSR row pointers, and conversion CSR -> ELL / DIA / BSR /
// COO plus the inverse (any format -> canonical COO).  Storage formats are
// those of the paper's Sec. 2.2 (ELL: rows packed to the longest row, stored
// column-major); conversion is what the runtime does when the chosen format
// differs from the one already held (Sec. 4).  Index work only: values are
// moved, never computed, so every output is bit-exact and deterministic.
#include <algorithm>
#include <cstdlib>
#include <cstring>

#include "gs_device.h"
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int kTB = 256;  // threads per block for the element-wise kernels

inline unsigned grid_for(int64_t n, int per_block = kTB)
{
    int64_t g = ceil_div(n, per_block);
    if (g < 1) g = 1;
    if (g > (1ll << 30)) g = 1ll << 30;
    return (unsigned)g;
}

#define GS_LAUNCH_CHECK() GS_HIP(hipGetLastError())

// ------------------------------------------------------------ validation

enum : int { kFlagIndex = 1, kFlagZero = 2, kFlagUnsorted = 4, kFlagDup = 8 };

// Entry k against its predecessor: index range, explicit zero, strict
// (row, col) order.
__device__ __forceinline__ int check_entry(int32_t r, int32_t c, float v, int32_t pr, int32_t pc, bool has_prev,
                                           int64_t R, int64_t C)
{
    int f = 0;
    if (r < 0 || r >= R || c < 0 || c >= C) f |= kFlagIndex;
    if (v == 0.0f) f |= kFlagZero;
    if (has_prev && !(pr < r || (pr == r && pc < c))) f |= kFlagUnsorted;
    return f;
}

// Validation flags of the COO, ORed into *flags (one atomic per workgroup at
// most, skipped when its bits are already set).  VEC: four entries per
// thread through 16-byte loads (all three arrays 16-byte aligned); the
// entries past the last whole quad are checked one by one.
template <bool VEC>
__global__ __launch_bounds__(kTB) void k_validate(const int32_t *__restrict__ row,
                                                  const int32_t *__restrict__ col,
                                                  const float *__restrict__ val, int64_t Z,
                                                  int64_t R, int64_t C, int *__restrict__ flags)
{
    __shared__ int red[kTB / kWave];
    int f = 0;
    const int64_t stride = (int64_t)gridDim.x * kTB;
    int64_t tail = 0;
    if (VEC) {
        const int64_t nq = Z / 4;
        for (int64_t q = (int64_t)blockIdx.x * kTB + threadIdx.x; q < nq; q += stride) {
            const int4 r4 = reinterpret_cast<const int4 *>(row)[q];
            const int4 c4 = reinterpret_cast<const int4 *>(col)[q];
            const float4 v4 = reinterpret_cast<const float4 *>(val)[q];
            const bool first = q == 0;
            const int32_t pr = first ? 0 : row[4 * q - 1], pc = first ? 0 : col[4 * q - 1];
            f |= check_entry(r4.x, c4.x, v4.x, pr, pc, !first, R, C);
            f |= check_entry(r4.y, c4.y, v4.y, r4.x, c4.x, true, R, C);
            f |= check_entry(r4.z, c4.z, v4.z, r4.y, c4.y, true, R, C);
            f |= check_entry(r4.w, c4.w, v4.w, r4.z, c4.z, true, R, C);
        }
        tail = nq * 4;
    }
    for (int64_t k = tail + (int64_t)blockIdx.x * kTB + threadIdx.x; k < Z; k += stride)
        f |= check_entry(row[k], col[k], val[k], k > 0 ? row[k - 1] : 0, k > 0 ? col[k - 1] : 0, k > 0, R, C);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) f |= __shfl_xor(f, o, kWave);
    if (lane_id() == 0) red[threadIdx.x / kWave] = f;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kTB / kWave; w++) f |= red[w];
        // the check may see a stale copy: then the (idempotent) atomic is issued
        if (f && (__hip_atomic_load(flags, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) & f) != f)
            atomicOr(flags, f);
    }
}

// ------------------------------------------------------------ radix sort
// LSD radix sort of the 64-bit keys (row << 32 | col), 8-bit digits, stable
// per pass, carrying the original position as payload.

constexpr int kRI = 16;             // keys per thread per tile
constexpr int kRT = kTB * kRI;      // keys per tile

__global__ __launch_bounds__(kTB) void k_make_keys(const int32_t *__restrict__ row,
                                                   const int32_t *__restrict__ col, int64_t Z,
                                                   uint64_t *__restrict__ keys)
{
    for (int64_t k = (int64_t)blockIdx.x * kTB + threadIdx.x; k < Z;
         k += (int64_t)gridDim.x * kTB)
        keys[k] = ((uint64_t)(uint32_t)row[k] << 32) | (uint32_t)col[k];
}

__global__ __launch_bounds__(kTB) void k_radix_hist(const uint64_t *__restrict__ keys, int64_t n,
                                                    int shift, int64_t ntiles,
                                                    int32_t *__restrict__ hist)
{
    __shared__ int h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kRT;
    for (int i = 0; i < kRI; i++) {
        int64_t k = base + (int64_t)i * kTB + threadIdx.x;
        if (k < n) atomicAdd(&h[(keys[k] >> shift) & 255], 1);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

__global__ __launch_bounds__(kTB) void k_radix_scatter(
    const uint64_t *__restrict__ kin, const uint32_t *__restrict__ pin, int64_t n, int shift,
    int64_t ntiles, const int32_t *__restrict__ off, uint64_t *__restrict__ kout,
    uint32_t *__restrict__ pout)
{
    constexpr int W = kTB / kWave;
    __shared__ int run[256];
    __shared__ int cnt[W][256];
    const int t = threadIdx.x, lane = t % kWave, w = t / kWave;
    run[t] = off[(int64_t)t * ntiles + blockIdx.x];
#pragma unroll
    for (int i = 0; i < W; i++) cnt[i][t] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kRT;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int r = 0; r < kRI; r++) {
        const int64_t k = base + (int64_t)r * kTB + t;
        const bool valid = k < n;
        const uint64_t key = valid ? kin[k] : 0ull;
        const int d = (int)((key >> shift) & 255);
        // lanes of this wave holding the same digit
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 8; bit++) {
            const uint64_t b = __ballot((d >> bit) & 1);
            peers &= ((d >> bit) & 1) ? b : ~b;
        }
        const int rank = __popcll(peers & lt);
        if (valid && rank == 0) cnt[w][d] = __popcll(peers);
        __syncthreads();
        if (valid) {
            int pos = run[d] + rank;
#pragma unroll
            for (int i = 0; i < W; i++)
                if (i < w) pos += cnt[i][d];
            kout[pos] = key;
            pout[pos] = pin ? pin[k] : (uint32_t)k;
        }
        __syncthreads();
        int add = 0;
#pragma unroll
        for (int i = 0; i < W; i++) {
            add += cnt[i][t];
            cnt[i][t] = 0;
        }
        run[t] += add;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kTB) void k_unpack_sorted(const uint64_t *__restrict__ keys,
                                                       const uint32_t *__restrict__ perm,
                                                       const float *__restrict__ val, int64_t Z,
                                                       int32_t *__restrict__ orow,
                                                       int32_t *__restrict__ ocol,
                                                       float *__restrict__ oval,
                                                       int *__restrict__ flags)
{
    int f = 0;
    for (int64_t k = (int64_t)blockIdx.x * kTB + threadIdx.x; k < Z;
         k += (int64_t)gridDim.x * kTB) {
        uint64_t key = keys[k];
        orow[k] = (int32_t)(key >> 32);
        ocol[k] = (int32_t)(key & 0xffffffffu);
        oval[k] = val[perm ? perm[k] : k];
        if (k > 0 && keys[k - 1] == key) f |= kFlagDup;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) f |= __shfl_xor(f, o, kWave);
    if (lane_id() == 0 && f) atomicOr(flags, f);
}


// ------------------------------------------------------------------- CSR

// row_ptr[i] = first position whose row is >= i: position k fills the
// pointers of every row in (row[k-1], row[k]].
// row_ptr from the sorted rows: the boundary between entries k-1 and k (k in
// [0, Z], with row -1 before the first entry and row R after the last)
// writes k into row_ptr of every row it starts.  Four boundaries per thread
// through one 16-byte load (row is the library's own 256-byte aligned buffer).
__global__ __launch_bounds__(kTB) void k_row_ptr(const int32_t *__restrict__ row, int64_t Z,
                                                 int64_t R, int32_t *__restrict__ row_ptr)
{
    const int64_t nq = Z / 4;
    const int64_t stride = (int64_t)gridDim.x * kTB;
    for (int64_t q = (int64_t)blockIdx.x * kTB + threadIdx.x; q < nq; q += stride) {
        const int4 r4 = reinterpret_cast<const int4 *>(row)[q];
        const int32_t rv[4] = {r4.x, r4.y, r4.z, r4.w};
        int64_t lo = q == 0 ? -1 : row[4 * q - 1];
#pragma unroll
        for (int j = 0; j < 4; j++) {
            for (int64_t i = lo + 1; i <= rv[j]; i++) row_ptr[i] = (int32_t)(4 * q + j);
            lo = rv[j];
        }
    }
    for (int64_t k = nq * 4 + (int64_t)blockIdx.x * kTB + threadIdx.x; k <= Z; k += stride) {
        const int64_t lo = (k == 0) ? -1 : row[k - 1];
        const int64_t hi = (k == Z) ? R : row[k];
        for (int64_t i = lo + 1; i <= hi; i++) row_ptr[i] = (int32_t)k;
    }
}

__global__ __launch_bounds__(kTB) void k_max_row_len(const int32_t *__restrict__ rp, int64_t R,
                                                     int *__restrict__ out)
{
    int m = 0;
    for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * kTB) {
        int n = rp[i + 1] - rp[i];
        m = n > m ? n : m;
    }
    m = wave_max_i32(m);
    if (lane_id() == 0 && m) atomicMax(out, m);
}

// ------------------------------------------------------------------- ELL

// Slot s = k*R + i (column-major): the k-th entry of row i or padding.
__global__ __launch_bounds__(kTB) void k_ell_fill(const int32_t *__restrict__ rp,
                                                  const int32_t *__restrict__ col,
                                                  const float *__restrict__ val, int64_t R,
                                                  int64_t K, int32_t *__restrict__ ec,
                                                  float *__restrict__ ev)
{
    const int64_t total = K * R;
    for (int64_t s = (int64_t)blockIdx.x * kTB + threadIdx.x; s < total;
         s += (int64_t)gridDim.x * kTB) {
        int64_t k = s / R, i = s - k * R;
        int64_t p = rp[i] + k;
        if (p < rp[i + 1]) {
            ec[s] = col[p];
            ev[s] = val[p];
        } else {
            ec[s] = -1;
            ev[s] = 0.0f;
        }
    }
}

// Row lengths of an ELL matrix: entries are packed to the front of a row.
__global__ __launch_bounds__(kTB) void k_ell_row_len(const int32_t *__restrict__ ec, int64_t R,
                                                     int64_t K, int32_t *__restrict__ len)
{
    for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * kTB) {
        int n = 0;
        for (int64_t k = 0; k < K; k++) {
            if (ec[k * R + i] == -1) break;
            n++;
        }
        len[i] = n;
    }
}

__global__ __launch_bounds__(kTB) void k_ell_to_coo(const int32_t *__restrict__ ec,
                                                    const float *__restrict__ ev, int64_t R,
                                                    int64_t K, const int32_t *__restrict__ pos,
                                                    int32_t *__restrict__ orow,
                                                    int32_t *__restrict__ ocol,
                                                    float *__restrict__ oval)
{
    const int64_t total = K * R;
    for (int64_t s = (int64_t)blockIdx.x * kTB + threadIdx.x; s < total;
         s += (int64_t)gridDim.x * kTB) {
        int64_t k = s / R, i = s - k * R;
        int32_t c = ec[s];
        if (c != -1) {
            int64_t p = pos[i] + k;
            orow[p] = (int32_t)i;
            ocol[p] = c;
            oval[p] = ev[s];
        }
    }
}

// Sum of cnt[0..n) (k_sum_counts) and number of BSR blocks with at least
// `thr` stored columns (k_count_dense): one partial per workgroup, or, from a
// one-workgroup grid, the result itself added to *out.
__global__ __launch_bounds__(kTB) void k_sum_counts(const int32_t *__restrict__ cnt, int64_t n,
                                                    unsigned long long *__restrict__ part,
                                                    unsigned long long *__restrict__ out)
{
    __shared__ unsigned long long t64[kTB / kWave];
    unsigned long long t = 0;
    for (int64_t k = (int64_t)blockIdx.x * kTB + threadIdx.x; k < n; k += (int64_t)gridDim.x * kTB)
        t += (unsigned long long)cnt[k];
    t = block_sum_u64<kTB>(t, t64);
    if (threadIdx.x != 0) return;
    if (gridDim.x == 1)
        *out += t;
    else
        part[blockIdx.x] = t;
}

__global__ __launch_bounds__(kTB) void k_count_dense(const uint64_t *__restrict__ mask, int64_t nb,
                                                     int thr, unsigned long long *__restrict__ part,
                                                     unsigned long long *__restrict__ out)
{
    __shared__ unsigned long long t64[kTB / kWave];
    unsigned long long n = 0;
    for (int64_t k = (int64_t)blockIdx.x * kTB + threadIdx.x; k < nb; k += (int64_t)gridDim.x * kTB)
        n += __popcll(mask[k]) >= thr;
    n = block_sum_u64<kTB>(n, t64);
    if (threadIdx.x != 0) return;
    if (gridDim.x == 1)
        *out += n;
    else
        part[blockIdx.x] = n;
}

inline unsigned reduce_grid(int64_t n)
{
    int64_t g = ceil_div(n, (int64_t)kTB * 4);
    return (unsigned)(g < 1 ? 1 : g > 2048 ? 2048 : g);
}

// ------------------------------------------------------------------- DIA
// Diagonal d of the R x C matrix has offset col - row in [-(R-1), C-1];
// slot index sidx = offset + R - 1.  A bitmap marks the occupied ones.

__global__ __launch_bounds__(kTB) void k_popc_words(const uint32_t *__restrict__ bm, int64_t nw,
                                                    int32_t *__restrict__ cnt)
{
    for (int64_t w = (int64_t)blockIdx.x * kTB + threadIdx.x; w < nw;
         w += (int64_t)gridDim.x * kTB)
        cnt[w] = __popc(bm[w]);
}

__global__ __launch_bounds__(kTB) void k_dia_offsets(const uint32_t *__restrict__ bm, int64_t nw,
                                                     const int32_t *__restrict__ wpos, int64_t R,
                                                     int32_t *__restrict__ offsets)
{
    for (int64_t w = (int64_t)blockIdx.x * kTB + threadIdx.x; w < nw;
         w += (int64_t)gridDim.x * kTB) {
        uint32_t bits = bm[w];
        int p = wpos[w];
        while (bits) {
            int b = __ffs(bits) - 1;
            bits &= bits - 1;
            offsets[p++] = (int32_t)(w * 32 + b - (R - 1));
        }
    }
}

__global__ __launch_bounds__(kTB) void k_dia_fill(const int32_t *__restrict__ row,
                                                  const int32_t *__restrict__ col,
                                                  const float *__restrict__ val, int64_t Z,
                                                  int64_t R, const uint32_t *__restrict__ bm,
                                                  const int32_t *__restrict__ wpos,
                                                  float *__restrict__ data)
{
    for (int64_t k = (int64_t)blockIdx.x * kTB + threadIdx.x; k < Z;
         k += (int64_t)gridDim.x * kTB) {
        int64_t sidx = (int64_t)col[k] - row[k] + R - 1;
        int64_t w = sidx >> 5;
        int64_t d = wpos[w] + __popc(bm[w] & ((1u << (sidx & 31)) - 1u));
        data[d * R + row[k]] = val[k];
    }
}

__global__ __launch_bounds__(kTB) void k_dia_row_len(const int32_t *__restrict__ offsets,
                                                     const float *__restrict__ data, int64_t ND,
                                                     int64_t R, int64_t C,
                                                     int32_t *__restrict__ len)
{
    for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * kTB) {
        int n = 0;
        for (int64_t d = 0; d < ND; d++) {
            int64_t j = i + offsets[d];
            if (j >= 0 && j < C && data[d * R + i] != 0.0f) n++;
        }
        len[i] = n;
    }
}

__global__ __launch_bounds__(kTB) void k_dia_to_coo(const int32_t *__restrict__ offsets,
                                                    const float *__restrict__ data, int64_t ND,
                                                    int64_t R, int64_t C,
                                                    const int32_t *__restrict__ pos,
                                                    int32_t *__restrict__ orow,
                                                    int32_t *__restrict__ ocol,
                                                    float *__restrict__ oval)
{
    for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * kTB) {
        int64_t p = pos[i];
        for (int64_t d = 0; d < ND; d++) {
            int64_t j = i + offsets[d];
            float v = data[d * R + i];
            if (j >= 0 && j < C && v != 0.0f) {
                orow[p] = (int32_t)i;
                ocol[p] = (int32_t)j;
                oval[p] = v;
                p++;
            }
        }
    }
}

// ------------------------------------------------------------------- BSR
// One wavefront per block row; lane l (< b) walks row br*b + l, whose
// columns are sorted, so its block columns arrive in ascending order.  The
// wave repeatedly takes the smallest pending block column over its lanes
// (a b-way merge): that is the next block of the block row.

__global__ __launch_bounds__(kTB) void k_bsr_count(const int32_t *__restrict__ rp,
                                                   const int32_t *__restrict__ col, int64_t R,
                                                   int b, int64_t nbr,
                                                   int32_t *__restrict__ cnt)
{
    const int64_t br = ((int64_t)blockIdx.x * kTB + threadIdx.x) / kWave;
    const int lane = lane_id();
    if (br >= nbr) return;  // whole wave leaves together
    const int64_t r = br * b + lane;
    int p = 0, e = 0;
    if (lane < b && r < R) {
        p = rp[r];
        e = rp[r + 1];
    }
    int n = 0;
    while (true) {
        int head = p < e ? col[p] / b : INT32_MAX;
        int m = wave_min_i32(head);
        if (m == INT32_MAX) break;
        n++;
        while (p < e && col[p] / b == m) p++;
    }
    if (lane == 0) cnt[br] = n;
}

// Block count with a bitmap of block columns in LDS (nbc bits), one
// workgroup per block row (persistent): the block row's entries are one
// contiguous range of col[], each sets its block column's bit, and the
// entries that found their bit clear count the distinct blocks.  The bitmap
// is zero at the top of every block row: after the count the touched words
// are cleared again by re-reading the entries when they are fewer than the
// bitmap's words (wide matrices: the whole-bitmap clear and population count
// had cost 267 us at 2M columns), the whole bitmap otherwise.
__global__ __launch_bounds__(kTB) void k_bsr_count_lds(const int32_t *__restrict__ rp,
                                                       const int32_t *__restrict__ col, int64_t R,
                                                       int b, int64_t nbr, int64_t nw,
                                                       int32_t *__restrict__ cnt)
{
    extern __shared__ uint32_t bmp[];
    __shared__ int wsum[kTB / kWave];
    for (int64_t w = threadIdx.x; w < nw; w += kTB) bmp[w] = 0u;
    __syncthreads();
    for (int64_t br = blockIdx.x; br < nbr; br += gridDim.x) {
        const int64_t r1 = (br + 1) * b < R ? (br + 1) * b : R;
        const int64_t k0 = rp[br * b], k1 = rp[r1];
        int n = 0;
        constexpr int U = 4;  // column loads in flight per thread (clamped indices: no branch per load)
        for (int64_t kb = k0 + threadIdx.x; kb < k1; kb += U * kTB) {
            int cv[U];
#pragma unroll
            for (int u = 0; u < U; u++) cv[u] = col[kb + u * kTB < k1 ? kb + u * kTB : k1 - 1];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const uint32_t c = (uint32_t)(cv[u] / b), bit = 1u << (c & 31);
                if (kb + u * kTB < k1) n += (atomicOr(&bmp[c >> 5], bit) & bit) ? 0 : 1;
            }
        }
        n = wave_sum_i32(n);
        if (lane_id() == 0) wsum[threadIdx.x / kWave] = n;
        __syncthreads();  // every bit of this block row is set and counted
        if (k1 - k0 < nw) {
            for (int64_t kk = k0 + threadIdx.x; kk < k1; kk += kTB) bmp[(uint32_t)(col[kk] / b) >> 5] = 0u;
        } else {
            for (int64_t w = threadIdx.x; w < nw; w += kTB) bmp[w] = 0u;
        }
        if (threadIdx.x == 0) {
            int t = 0;
            for (int i = 0; i < kTB / kWave; i++) t += wsum[i];
            cnt[br] = t;
        }
        __syncthreads();  // the bitmap is clear and wsum read before the next block row
    }
}

// BSR fill with a bitmap of block columns in LDS, one workgroup per block
// row (persistent).  The block row's entries mark their block columns; an
// exclusive prefix of the bitmap words' populations numbers the blocks in
// column order (block j of the row is the j-th set bit), which gives bcol
// and, for every entry, its block: the entries are placed in parallel, so a
// block row holding a hub row costs its entries, not one step per block.
// bmask must be zero on entry.
__global__ __launch_bounds__(kTB) void k_bsr_fill_lds(const int32_t *__restrict__ rp,
                                                      const int32_t *__restrict__ col,
                                                      const float *__restrict__ val, int64_t R, int b,
                                                      int64_t nbr, int64_t nw,
                                                      const int32_t *__restrict__ bptr,
                                                      int32_t *__restrict__ bcol,
                                                      float *__restrict__ bval,
                                                      unsigned long long *__restrict__ bmask)
{
    extern __shared__ uint32_t sm[];
    uint32_t *bmp = sm;                                   // nw words
    int32_t *pre = reinterpret_cast<int32_t *>(sm + nw);  // nw prefix counts
    __shared__ int32_t lrp[65];                           // the block row's row pointers (b <= 64)
    __shared__ int tmp[kTB / kWave];
    __shared__ int carry;
    const int64_t bb = (int64_t)b * b;
    for (int64_t br = blockIdx.x; br < nbr; br += gridDim.x) {
        const int64_t r0 = br * b;
        const int nr = (int)(R - r0 < b ? R - r0 : b);
        for (int64_t w = threadIdx.x; w < nw; w += kTB) bmp[w] = 0u;
        if (threadIdx.x <= nr) lrp[threadIdx.x] = rp[r0 + threadIdx.x];
        if (threadIdx.x == 0) carry = 0;
        __syncthreads();
        const int64_t k0 = lrp[0], k1 = lrp[nr];
        for (int64_t k = k0 + threadIdx.x; k < k1; k += kTB) {
            const uint32_t c = (uint32_t)(col[k] / b);
            atomicOr(&bmp[c >> 5], 1u << (c & 31));
        }
        __syncthreads();
        for (int64_t w0 = 0; w0 < nw; w0 += kTB) {
            const int64_t w = w0 + threadIdx.x;
            const int pc = w < nw ? __popc(bmp[w]) : 0;
            const int ex = block_exclusive_scan<kTB>(pc, tmp);
            const int base = carry;
            if (w < nw) pre[w] = base + ex;
            __syncthreads();
            if (threadIdx.x == kTB - 1) carry = base + ex + pc;
            __syncthreads();
        }
        const int64_t blk0 = bptr[br];
        for (int64_t w = threadIdx.x; w < nw; w += kTB) {
            uint32_t x = bmp[w];
            int64_t n = blk0 + pre[w];
            while (x) {
                bcol[n++] = (int32_t)(w * 32 + __ffs(x) - 1);
                x &= x - 1;
            }
        }
        for (int64_t k = k0 + threadIdx.x; k < k1; k += kTB) {
            int lo = 0, hi = nr - 1;  // row of entry k: last li with lrp[li] <= k
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (lrp[mid] <= k)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            const int c = col[k];
            const uint32_t bc = (uint32_t)(c / b);
            const int64_t blk = blk0 + pre[bc >> 5] + __popc(bmp[bc >> 5] & ((1u << (bc & 31)) - 1u));
            const int cc = c - (int)bc * b;
            bval[blk * bb + (int64_t)lo * b + cc] = val[k];
            atomicOr(&bmask[blk], 1ull << cc);
        }
        __syncthreads();  // before the next block row reuses the LDS
    }
}

__global__ __launch_bounds__(kTB) void k_bsr_fill(const int32_t *__restrict__ rp,
                                                  const int32_t *__restrict__ col,
                                                  const float *__restrict__ val, int64_t R, int b,
                                                  int64_t nbr, const int32_t *__restrict__ bptr,
                                                  int32_t *__restrict__ bcol,
                                                  float *__restrict__ bval,
                                                  uint64_t *__restrict__ bmask)
{
    const int64_t br = ((int64_t)blockIdx.x * kTB + threadIdx.x) / kWave;
    const int lane = lane_id();
    if (br >= nbr) return;
    const int64_t r = br * b + lane;
    int p = 0, e = 0;
    if (lane < b && r < R) {
        p = rp[r];
        e = rp[r + 1];
    }
    int64_t blk = bptr[br];
    const int64_t bb = (int64_t)b * b;
    while (true) {
        int head = p < e ? col[p] / b : INT32_MAX;
        int m = wave_min_i32(head);
        if (m == INT32_MAX) break;
        uint64_t mask = 0;
        while (p < e && col[p] / b == m) {
            int cc = col[p] - m * b;
            bval[blk * bb + (int64_t)lane * b + cc] = val[p];
            mask |= 1ull << cc;
            p++;
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) mask |= __shfl_xor(mask, o, kWave);
        if (lane == 0) {
            bcol[blk] = m;
            bmask[blk] = mask;
        }
        blk++;
    }
}

__global__ __launch_bounds__(kTB) void k_bsr_row_len(const int32_t *__restrict__ bptr,
                                                     const int32_t *__restrict__ bcol,
                                                     const float *__restrict__ bval, int64_t R,
                                                     int64_t C, int b,
                                                     int32_t *__restrict__ len)
{
    const int64_t bb = (int64_t)b * b;
    for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * kTB) {
        int64_t br = i / b, ii = i - br * b;
        int n = 0;
        for (int64_t blk = bptr[br]; blk < bptr[br + 1]; blk++)
            for (int jj = 0; jj < b; jj++) {
                int64_t j = (int64_t)bcol[blk] * b + jj;
                if (j < C && bval[blk * bb + ii * b + jj] != 0.0f) n++;
            }
        len[i] = n;
    }
}

__global__ __launch_bounds__(kTB) void k_bsr_to_coo(const int32_t *__restrict__ bptr,
                                                    const int32_t *__restrict__ bcol,
                                                    const float *__restrict__ bval, int64_t R,
                                                    int64_t C, int b,
                                                    const int32_t *__restrict__ pos,
                                                    int32_t *__restrict__ orow,
                                                    int32_t *__restrict__ ocol,
                                                    float *__restrict__ oval)
{
    const int64_t bb = (int64_t)b * b;
    for (int64_t i = (int64_t)blockIdx.x * kTB + threadIdx.x; i < R;
         i += (int64_t)gridDim.x * kTB) {
        int64_t br = i / b, ii = i - br * b;
        int64_t p = pos[i];
        for (int64_t blk = bptr[br]; blk < bptr[br + 1]; blk++)
            for (int jj = 0; jj < b; jj++) {
                int64_t j = (int64_t)bcol[blk] * b + jj;
                float v = bval[blk * bb + ii * b + jj];
                if (j < C && v != 0.0f) {
                    orow[p] = (int32_t)i;
                    ocol[p] = (int32_t)j;
                    oval[p] = v;
                    p++;
                }
            }
    }
}

// ------------------------------------------------------------ CSR -> COO

// Row index of every entry: groups of 8 lanes per row, so a long row is
// written by 8 lanes side by side and a wave covers 8 rows at once.
__global__ __launch_bounds__(kTB) void k_expand_rows(const int32_t *__restrict__ rp, int64_t R,
                                                     int32_t *__restrict__ orow)
{
    constexpr int G = 8;
    const int lane = threadIdx.x % G;
    const int64_t groups = (int64_t)gridDim.x * (kTB / G);
    for (int64_t i = ((int64_t)blockIdx.x * kTB + threadIdx.x) / G; i < R; i += groups)
        for (int64_t k = rp[i] + lane; k < rp[i + 1]; k += G) orow[k] = (int32_t)i;
}


// Distinct (row/b, col/b) blocks per block row into cnt[0..nbr).  The LDS
// bitmap kernel needs nbc/8 bytes of LDS; wider matrices use the merge (the
// BSR fill makes the same choice).
void launch_block_count(const int32_t *rp, const int32_t *col, int64_t R, int64_t C, int b,
                        int64_t nbr, int32_t *cnt, hipStream_t s)
{
    const int64_t nbc = ceil_div(C, b), nw = ceil_div(nbc, 32);
    const char *force_merge = std::getenv("GS_BLOCK_COUNT_MERGE");
    if (nw * 4 <= 48 * 1024 && !(force_merge && *force_merge == '1')) {
        const int64_t g = std::min<int64_t>(nbr, 256 * 8);
        k_bsr_count_lds<<<(unsigned)std::max<int64_t>(1, g), kTB, (size_t)nw * 4, s>>>(rp, col, R, b, nbr, nw, cnt);
    } else {
        k_bsr_count<<<grid_for(nbr * kWave), kTB, 0, s>>>(rp, col, R, b, nbr, cnt);
    }
    GS_LAUNCH_CHECK();
}

int read_flag(const int *d_flags, hipStream_t s)
{
    int h = 0;
    GS_HIP(hipMemcpyAsync(&h, d_flags, sizeof(int), hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));
    return h;
}

inline unsigned elem_grid(int64_t n)
{
    // grid-stride kernels: enough blocks to fill 256 CUs several times over
    int64_t g = ceil_div(n, kTB);
    if (g > 256 * 64) g = 256 * 64;
    if (g < 1) g = 1;
    return (unsigned)g;
}

}  // namespace

// ======================================================================

int bits_for(int64_t maxval)
{
    int b = 0;
    while (b < 63 && (1ll << b) <= maxval) b++;
    return b;
}

void radix_sort_pairs(uint64_t *ka, uint64_t *kb, uint32_t *pa, uint32_t *pb, int64_t n,
                      const std::vector<int> &shifts, hipStream_t s, uint64_t **keys,
                      uint32_t **perm)
{
    uint64_t *kin = ka, *kout = kb;
    uint32_t *pin = nullptr, *pout = pa, *pspare = pb;
    if (n > 0 && !shifts.empty()) {
        const int64_t ntiles = ceil_div(n, kRT);
        DevBuf hist;
        hist.alloc((size_t)(256 * ntiles + 1) * 4, s);
        for (size_t i = 0; i < shifts.size(); i++) {
            k_radix_hist<<<(unsigned)ntiles, kTB, 0, s>>>(kin, n, shifts[i], ntiles, hist.as<int32_t>());
            GS_LAUNCH_CHECK();
            exclusive_scan_i32(hist.as<int32_t>(), hist.as<int32_t>(), 256 * ntiles, false, s);
            k_radix_scatter<<<(unsigned)ntiles, kTB, 0, s>>>(kin, pin, n, shifts[i], ntiles,
                                                             hist.as<int32_t>(), kout, pout);
            GS_LAUNCH_CHECK();
            std::swap(kin, kout);
            uint32_t *used = pout;
            pout = (pin == nullptr) ? pspare : pin;
            pin = used;
        }
    }
    *keys = kin;
    *perm = pin;
}

// Sorts the triplets (major[k], minor[k], val[k]) by (major, minor) into
// omajor / ominor / oval (a stable LSD radix sort over the bits in use).
// Used to move between row-major and column-major orders.
void sort_triplets(const int32_t *major, const int32_t *minor, const float *val, int64_t Z,
                   int64_t n_major, int64_t n_minor, int32_t *omajor, int32_t *ominor, float *oval,
                   hipStream_t s)
{
    if (Z == 0) return;
    std::vector<int> shifts;
    for (int sft = 0; sft < bits_for(n_minor - 1); sft += 8) shifts.push_back(sft);
    for (int sft = 0; sft < bits_for(n_major - 1); sft += 8) shifts.push_back(32 + sft);
    DevBuf k0, k1, p0, p1, flags;
    k0.alloc((size_t)Z * 8, s);
    k1.alloc((size_t)Z * 8, s);
    p0.alloc((size_t)Z * 4, s);
    p1.alloc((size_t)Z * 4, s);
    flags.alloc(sizeof(int), s);
    GS_HIP(hipMemsetAsync(flags.p, 0, sizeof(int), s));
    k_make_keys<<<elem_grid(Z), kTB, 0, s>>>(major, minor, Z, k0.as<uint64_t>());
    GS_LAUNCH_CHECK();
    uint64_t *keys = nullptr;
    uint32_t *perm = nullptr;
    radix_sort_pairs(k0.as<uint64_t>(), k1.as<uint64_t>(), p0.as<uint32_t>(), p1.as<uint32_t>(), Z,
                     shifts, s, &keys, &perm);
    k_unpack_sorted<<<elem_grid(Z), kTB, 0, s>>>(keys, perm, val, Z, omajor, ominor, oval,
                                                 flags.as<int>());
    GS_LAUNCH_CHECK();
}

void canonicalize(const gs_coo &A, bool assume_canonical, hipStream_t s, CanonCOO &out)
{
    const int64_t R = A.n_rows, C = A.n_cols, Z = A.nnz;
    out.R = R;
    out.C = C;
    out.Z = Z;
    out.row.alloc((size_t)Z * 4, s);
    out.col.alloc((size_t)Z * 4, s);
    out.val.alloc((size_t)Z * 4, s);
    if (Z == 0) return;

    DevBuf flags;
    flags.alloc(sizeof(int), s);
    GS_HIP(hipMemsetAsync(flags.p, 0, sizeof(int), s));
    const bool aligned = ((reinterpret_cast<uintptr_t>(A.row) | reinterpret_cast<uintptr_t>(A.col) |
                           reinterpret_cast<uintptr_t>(A.val)) & 15) == 0;
    if (aligned)
        k_validate<true><<<elem_grid(ceil_div(Z, 4)), kTB, 0, s>>>(A.row, A.col, A.val, Z, R, C, flags.as<int>());
    else
        k_validate<false><<<elem_grid(Z), kTB, 0, s>>>(A.row, A.col, A.val, Z, R, C, flags.as<int>());
    GS_LAUNCH_CHECK();
    int f = read_flag(flags.as<int>(), s);
    if (f & kFlagIndex) fail(GS_ERR_INDEX, "COO index outside the %lld x %lld matrix", (long long)R, (long long)C);
    if (f & kFlagZero) fail(GS_ERR_EXPLICIT_ZERO, "COO holds an explicit zero value");
    if (!(f & kFlagUnsorted)) {
        GS_HIP(hipMemcpyAsync(out.row.p, A.row, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
        GS_HIP(hipMemcpyAsync(out.col.p, A.col, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
        GS_HIP(hipMemcpyAsync(out.val.p, A.val, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
        return;
    }
    if (assume_canonical)
        fail(GS_ERR_INVALID_ARG, "assume_canonical set but the COO is not strictly (row,col)-sorted");

    // LSD radix sort over the bits that are in use.
    const int bc = bits_for(C - 1), br = bits_for(R - 1);
    std::vector<int> shifts;
    for (int sft = 0; sft < bc; sft += 8) shifts.push_back(sft);
    for (int sft = 0; sft < br; sft += 8) shifts.push_back(32 + sft);
    DevBuf k0, k1, p0, p1;
    k0.alloc((size_t)Z * 8, s);
    k1.alloc((size_t)Z * 8, s);
    p0.alloc((size_t)Z * 4, s);
    p1.alloc((size_t)Z * 4, s);
    k_make_keys<<<elem_grid(Z), kTB, 0, s>>>(A.row, A.col, Z, k0.as<uint64_t>());
    GS_LAUNCH_CHECK();
    uint64_t *kin = nullptr;
    uint32_t *pin = nullptr;
    radix_sort_pairs(k0.as<uint64_t>(), k1.as<uint64_t>(), p0.as<uint32_t>(), p1.as<uint32_t>(), Z,
                     shifts, s, &kin, &pin);
    GS_HIP(hipMemsetAsync(flags.p, 0, sizeof(int), s));
    k_unpack_sorted<<<elem_grid(Z), kTB, 0, s>>>(kin, pin, A.val, Z, out.row.as<int32_t>(),
                                                 out.col.as<int32_t>(), out.val.as<float>(),
                                                 flags.as<int>());
    GS_LAUNCH_CHECK();
    f = read_flag(flags.as<int>(), s);  // also keeps the sort buffers alive until done
    if (f & kFlagDup) fail(GS_ERR_DUPLICATE, "COO holds duplicate (row, col) entries");
}

gs_matrix_ *csr_from_canon(CanonCOO &&c, hipStream_t s, bool plan)
{
    gs_matrix_ *m = new gs_matrix_();
    try {
        m->fmt = GS_CSR;
        m->R = c.R;
        m->C = c.C;
        m->Z = c.Z;
        m->stream = s;
        m->row_ptr.alloc((size_t)(c.R + 1) * 4, s);
        k_row_ptr<<<elem_grid(ceil_div(c.Z, 4) + 1), kTB, 0, s>>>(c.row.as<int32_t>(), c.Z, c.R,
                                                     m->row_ptr.as<int32_t>());
        GS_LAUNCH_CHECK();
        m->col = std::move(c.col);
        m->val = std::move(c.val);
        m->device_bytes = (uint64_t)(c.R + 1) * 4 + (uint64_t)c.Z * 8;
        if (plan) plan_csr(*m, s);
    } catch (...) {
        delete m;
        throw;
    }
    return m;
}

uint64_t format_bytes(int fmt, int64_t R, int64_t C, int64_t Z, int64_t K, int64_t ND, int64_t nb,
                      int b)
{
    switch (fmt) {
    case GS_COO: return (uint64_t)Z * 12;
    case GS_CSR: return (uint64_t)(R + 1) * 4 + (uint64_t)Z * 8;
    case GS_CSC: return (uint64_t)(C + 1) * 4 + (uint64_t)Z * 8;
    case GS_ELL: return (uint64_t)K * (uint64_t)R * 8;
    case GS_DIA: return (uint64_t)ND * 4 + (uint64_t)ND * (uint64_t)R * 4;
    case GS_BSR: {
        int64_t nbr = ceil_div(R, b);
        return (uint64_t)(nbr + 1) * 4 + (uint64_t)nb * (4 + 8) + (uint64_t)nb * b * b * 4;
    }
    }
    return 0;
}

void count_blocks_async(const gs_matrix_ &csr, int b, unsigned long long *total, hipStream_t s)
{
    const int64_t nbr = ceil_div(csr.R, b);
    if (nbr == 0 || csr.Z == 0) return;
    DevBuf cnt;
    cnt.alloc((size_t)nbr * 4, s);
    launch_block_count(csr.row_ptr.as<int32_t>(), csr.col.as<int32_t>(), csr.R, csr.C, b, nbr,
                       cnt.as<int32_t>(), s);
    const unsigned G = reduce_grid(nbr);
    DevBuf part;
    if (G > 1) part.alloc(sizeof(unsigned long long) * G, s);
    k_sum_counts<<<G, kTB, 0, s>>>(cnt.as<int32_t>(), nbr, part.as<unsigned long long>(), total);
    GS_LAUNCH_CHECK();
    if (G > 1) add_partials_u64(part.as<unsigned long long>(), G, total, s);
}

int64_t count_blocks(const gs_matrix_ &csr, int b, hipStream_t s)
{
    DevBuf d;
    d.alloc(sizeof(unsigned long long), s);
    GS_HIP(hipMemsetAsync(d.p, 0, sizeof(unsigned long long), s));
    count_blocks_async(csr, b, d.as<unsigned long long>(), s);
    unsigned long long nb = 0;
    GS_HIP(hipMemcpyAsync(&nb, d.p, sizeof nb, hipMemcpyDeviceToHost, s));
    GS_HIP(hipStreamSynchronize(s));
    return (int64_t)nb;
}

gs_matrix_ *convert_from_csr(const gs_matrix_ &csr, int fmt, int bsr_block, uint64_t max_bytes,
                             hipStream_t s, uint64_t *bytes_required)
{
    const int64_t R = csr.R, C = csr.C, Z = csr.Z;
    const int32_t *rp = csr.row_ptr.as<int32_t>();
    const int32_t *col = csr.col.as<int32_t>();
    const float *val = csr.val.as<float>();
    gs_matrix_ *m = new gs_matrix_();
    try {
        m->fmt = fmt;
        m->R = R;
        m->C = C;
        m->Z = Z;
        m->stream = s;
        switch (fmt) {
        case GS_CSR: {
            uint64_t need = format_bytes(GS_CSR, R, C, Z, 0, 0, 0, 0);
            if (bytes_required) *bytes_required = need;
            m->row_ptr.alloc((size_t)(R + 1) * 4, s);
            m->col.alloc((size_t)Z * 4, s);
            m->val.alloc((size_t)Z * 4, s);
            GS_HIP(hipMemcpyAsync(m->row_ptr.p, rp, (size_t)(R + 1) * 4, hipMemcpyDeviceToDevice, s));
            if (Z) {
                GS_HIP(hipMemcpyAsync(m->col.p, col, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
                GS_HIP(hipMemcpyAsync(m->val.p, val, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
            }
            m->device_bytes = need;
            plan_csr(*m, s);
            break;
        }
        case GS_CSC: {
            uint64_t need = format_bytes(GS_CSC, R, C, Z, 0, 0, 0, 0);
            if (bytes_required) *bytes_required = need;
            m->row_ptr.alloc((size_t)(C + 1) * 4, s);
            m->col.alloc((size_t)Z * 4, s);
            m->val.alloc((size_t)Z * 4, s);
            DevBuf rows, cols;
            rows.alloc((size_t)Z * 4, s);
            cols.alloc((size_t)Z * 4, s);
            if (Z) {
                k_expand_rows<<<elem_grid(R * 8), kTB, 0, s>>>(rp, R, rows.as<int32_t>());
                GS_LAUNCH_CHECK();
                sort_triplets(col, rows.as<int32_t>(), val, Z, C, R, cols.as<int32_t>(),
                              m->col.as<int32_t>(), m->val.as<float>(), s);
            }
            k_row_ptr<<<elem_grid(ceil_div(Z, 4) + 1), kTB, 0, s>>>(cols.as<int32_t>(), Z, C, m->row_ptr.as<int32_t>());
            GS_LAUNCH_CHECK();
            m->device_bytes = need;
            break;
        }
        case GS_COO: {
            uint64_t need = format_bytes(GS_COO, R, C, Z, 0, 0, 0, 0);
            if (bytes_required) *bytes_required = need;
            m->row.alloc((size_t)Z * 4, s);
            m->col.alloc((size_t)Z * 4, s);
            m->val.alloc((size_t)Z * 4, s);
            if (Z) {
                k_expand_rows<<<elem_grid(R * 8), kTB, 0, s>>>(rp, R, m->row.as<int32_t>());
                GS_LAUNCH_CHECK();
                GS_HIP(hipMemcpyAsync(m->col.p, col, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
                GS_HIP(hipMemcpyAsync(m->val.p, val, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
            }
            m->device_bytes = need;
            plan_coo(*m, rp, s);
            break;
        }
        case GS_ELL: {
            DevBuf mx;
            mx.alloc(sizeof(int), s);
            GS_HIP(hipMemsetAsync(mx.p, 0, sizeof(int), s));
            if (R) {
                // a few hundred workgroups: one atomic per wave on one word
                k_max_row_len<<<(unsigned)std::min<int64_t>(256, ceil_div(R, kTB)), kTB, 0, s>>>(
                    rp, R, mx.as<int>());
                GS_LAUNCH_CHECK();
            }
            m->K = read_flag(mx.as<int>(), s);
            uint64_t need = format_bytes(GS_ELL, R, C, Z, m->K, 0, 0, 0);
            if (bytes_required) *bytes_required = need;
            if (need > max_bytes)
                fail(GS_ERR_INFEASIBLE, "ELL needs %llu bytes (K=%lld), over the cap of %llu",
                     (unsigned long long)need, (long long)m->K, (unsigned long long)max_bytes);
            m->ell_col.alloc((size_t)(m->K * R) * 4, s);
            m->ell_val.alloc((size_t)(m->K * R) * 4, s);
            if (m->K * R) {
                k_ell_fill<<<elem_grid(m->K * R), kTB, 0, s>>>(rp, col, val, R, m->K,
                                                               m->ell_col.as<int32_t>(),
                                                               m->ell_val.as<float>());
                GS_LAUNCH_CHECK();
            }
            m->device_bytes = need;
            // row tiles whose X window the SpMM may stage in LDS (rows of one chain only)
            if (const char *e = std::getenv("GS_ELL_WINDOW"); Z > 0 && m->K <= kChainFold && !(e && std::string(e) == "off"))
                count_windows(*m, rp, col, s);
            break;
        }
        case GS_DIA: {
            const int64_t span = (R > 0 && C > 0) ? R + C - 1 : 0;
            const int64_t nw = ceil_div(span, 32);
            DevBuf bm, wpos, row;
            bm.alloc((size_t)(nw + 1) * 4, s);
            wpos.alloc((size_t)(nw + 1) * 4, s);
            row.alloc((size_t)Z * 4, s);
            if (Z) {
                k_expand_rows<<<elem_grid(R * 8), kTB, 0, s>>>(rp, R, row.as<int32_t>());
                GS_LAUNCH_CHECK();
                diag_bitmap(rp, col, R, C, Z, bm.as<uint32_t>(), s);
                k_popc_words<<<elem_grid(nw), kTB, 0, s>>>(bm.as<uint32_t>(), nw, wpos.as<int32_t>());
                GS_LAUNCH_CHECK();
                exclusive_scan_i32(wpos.as<int32_t>(), wpos.as<int32_t>(), nw, true, s);
                int32_t nd = 0;
                GS_HIP(hipMemcpyAsync(&nd, wpos.as<int32_t>() + nw, 4, hipMemcpyDeviceToHost, s));
                GS_HIP(hipStreamSynchronize(s));
                m->ND = nd;
            }
            uint64_t need = format_bytes(GS_DIA, R, C, Z, 0, m->ND, 0, 0);
            if (bytes_required) *bytes_required = need;
            if (need > max_bytes)
                fail(GS_ERR_INFEASIBLE, "DIA needs %llu bytes (%lld diagonals), over the cap of %llu",
                     (unsigned long long)need, (long long)m->ND, (unsigned long long)max_bytes);
            m->offsets.alloc((size_t)m->ND * 4, s);
            m->dia.alloc((size_t)(m->ND * R) * 4, s);
            if (Z) {
                k_dia_offsets<<<elem_grid(nw), kTB, 0, s>>>(bm.as<uint32_t>(), nw, wpos.as<int32_t>(),
                                                             R, m->offsets.as<int32_t>());
                GS_LAUNCH_CHECK();
                GS_HIP(hipMemsetAsync(m->dia.p, 0, (size_t)(m->ND * R) * 4, s));
                k_dia_fill<<<elem_grid(Z), kTB, 0, s>>>(row.as<int32_t>(), col, val, Z, R,
                                                        bm.as<uint32_t>(), wpos.as<int32_t>(),
                                                        m->dia.as<float>());
                GS_LAUNCH_CHECK();
            }
            m->device_bytes = need;
            break;
        }
        case GS_BSR: {
            const int b = bsr_block;
            if (b < 1 || b > 64) fail(GS_ERR_INVALID_ARG, "BSR block size %d outside 1..64", b);
            m->b = b;
            const int64_t nbr = ceil_div(R, b);
            DevBuf cnt;
            cnt.alloc((size_t)(nbr + 1) * 4, s);
            if (nbr) launch_block_count(rp, col, R, C, b, nbr, cnt.as<int32_t>(), s);
            exclusive_scan_i32(cnt.as<int32_t>(), cnt.as<int32_t>(), nbr, true, s);
            int32_t nb = 0;
            GS_HIP(hipMemcpyAsync(&nb, cnt.as<int32_t>() + nbr, 4, hipMemcpyDeviceToHost, s));
            GS_HIP(hipStreamSynchronize(s));
            m->nb = nb;
            uint64_t need = format_bytes(GS_BSR, R, C, Z, 0, 0, nb, b);
            if (bytes_required) *bytes_required = need;
            if (need > max_bytes)
                fail(GS_ERR_INFEASIBLE, "BSR(%d) needs %llu bytes (%lld blocks), over the cap of %llu",
                     b, (unsigned long long)need, (long long)nb, (unsigned long long)max_bytes);
            m->bptr = std::move(cnt);
            m->bcol.alloc((size_t)nb * 4, s);
            m->bmask.alloc((size_t)nb * 8, s);
            m->bval.alloc((size_t)nb * b * b * 4, s);
            if (nb) {
                GS_HIP(hipMemsetAsync(m->bval.p, 0, (size_t)nb * b * b * 4, s));
                const int64_t nw = ceil_div(ceil_div(C, b), 32);
                const size_t lds = (size_t)nw * 8;  // bitmap + prefix counts
                const char *force_merge = std::getenv("GS_BLOCK_COUNT_MERGE");
                if ((int64_t)lds + 2048 <= max_lds_bytes() && !(force_merge && *force_merge == '1')) {
                    GS_HIP(hipMemsetAsync(m->bmask.p, 0, (size_t)nb * 8, s));
                    k_bsr_fill_lds<<<(unsigned)std::min<int64_t>(nbr, 256 * 8), kTB, lds, s>>>(
                        rp, col, val, R, b, nbr, nw, m->bptr.as<int32_t>(), m->bcol.as<int32_t>(),
                        m->bval.as<float>(), m->bmask.as<unsigned long long>());
                } else {
                    k_bsr_fill<<<grid_for(nbr * kWave), kTB, 0, s>>>(
                        rp, col, val, R, b, nbr, m->bptr.as<int32_t>(), m->bcol.as<int32_t>(),
                        m->bval.as<float>(), m->bmask.as<uint64_t>());
                }
                GS_LAUNCH_CHECK();
                // dense-block count (kernel choice at SpMM time)
                DevBuf dn;
                dn.alloc(sizeof(unsigned long long), s);
                GS_HIP(hipMemsetAsync(dn.p, 0, sizeof(unsigned long long), s));
                const unsigned G = reduce_grid(nb);
                DevBuf part;
                if (G > 1) part.alloc(sizeof(unsigned long long) * G, s);
                k_count_dense<<<G, kTB, 0, s>>>(m->bmask.as<uint64_t>(), nb, kBsrDenseCols,
                                                part.as<unsigned long long>(), dn.as<unsigned long long>());
                GS_LAUNCH_CHECK();
                if (G > 1) add_partials_u64(part.as<unsigned long long>(), G, dn.as<unsigned long long>(), s);
                unsigned long long dense = 0;
                GS_HIP(hipMemcpyAsync(&dense, dn.p, sizeof dense, hipMemcpyDeviceToHost, s));
                GS_HIP(hipStreamSynchronize(s));
                m->n_dense_blocks = (int64_t)dense;
                plan_bsr_hybrid(*m, rp, col, val, s);
            }
            m->device_bytes = need;
            break;
        }
        default: fail(GS_ERR_INVALID_ARG, "unknown format %d", fmt);
        }
        GS_HIP(hipStreamSynchronize(s));
    } catch (...) {
        delete m;
        throw;
    }
    return m;
}

void to_coo(const gs_matrix_ &m, int32_t *row, int32_t *col, float *val, hipStream_t s)
{
    const int64_t R = m.R, C = m.C, Z = m.Z;
    if (Z == 0) return;
    switch (m.fmt) {
    case GS_COO:
        GS_HIP(hipMemcpyAsync(row, m.row.p, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
        GS_HIP(hipMemcpyAsync(col, m.col.p, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
        GS_HIP(hipMemcpyAsync(val, m.val.p, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
        return;
    case GS_CSR:
        k_expand_rows<<<elem_grid(R * 8), kTB, 0, s>>>(m.row_ptr.as<int32_t>(), R, row);
        GS_LAUNCH_CHECK();
        GS_HIP(hipMemcpyAsync(col, m.col.p, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
        GS_HIP(hipMemcpyAsync(val, m.val.p, (size_t)Z * 4, hipMemcpyDeviceToDevice, s));
        return;
    case GS_CSC: {  // back to (row, col) order
        DevBuf cols;
        cols.alloc((size_t)Z * 4, s);
        k_expand_rows<<<elem_grid(C * 8), kTB, 0, s>>>(m.row_ptr.as<int32_t>(), C, cols.as<int32_t>());
        GS_LAUNCH_CHECK();
        sort_triplets(m.col.as<int32_t>(), cols.as<int32_t>(), m.val.as<float>(), Z, R, C, row, col,
                      val, s);
        return;
    }
    default: break;
    }
    DevBuf pos;
    pos.alloc((size_t)(R + 1) * 4, s);
    int32_t *p = pos.as<int32_t>();
    switch (m.fmt) {
    case GS_ELL:
        k_ell_row_len<<<elem_grid(R), kTB, 0, s>>>(m.ell_col.as<int32_t>(), R, m.K, p);
        GS_LAUNCH_CHECK();
        exclusive_scan_i32(p, p, R, true, s);
        k_ell_to_coo<<<elem_grid(m.K * R), kTB, 0, s>>>(m.ell_col.as<int32_t>(), m.ell_val.as<float>(),
                                                        R, m.K, p, row, col, val);
        break;
    case GS_DIA:
        k_dia_row_len<<<elem_grid(R), kTB, 0, s>>>(m.offsets.as<int32_t>(), m.dia.as<float>(), m.ND,
                                                   R, C, p);
        GS_LAUNCH_CHECK();
        exclusive_scan_i32(p, p, R, true, s);
        k_dia_to_coo<<<elem_grid(R), kTB, 0, s>>>(m.offsets.as<int32_t>(), m.dia.as<float>(), m.ND,
                                                  R, C, p, row, col, val);
        break;
    case GS_BSR:
        k_bsr_row_len<<<elem_grid(R), kTB, 0, s>>>(m.bptr.as<int32_t>(), m.bcol.as<int32_t>(),
                                                   m.bval.as<float>(), R, C, m.b, p);
        GS_LAUNCH_CHECK();
        exclusive_scan_i32(p, p, R, true, s);
        k_bsr_to_coo<<<elem_grid(R), kTB, 0, s>>>(m.bptr.as<int32_t>(), m.bcol.as<int32_t>(),
                                                  m.bval.as<float>(), R, C, m.b, p, row, col, val);
        break;
    default: fail(GS_ERR_INVALID_ARG, "corrupt matrix handle");
    }
    GS_LAUNCH_CHECK();
}

gs_matrix_ *csr_from_any(const gs_matrix_ &m, hipStream_t s)
{
    if (m.fmt == GS_CSR) return convert_from_csr(m, GS_CSR, 0, ~0ull, s, nullptr);
    CanonCOO c;
    c.R = m.R;
    c.C = m.C;
    c.Z = m.Z;
    c.row.alloc((size_t)m.Z * 4, s);
    c.col.alloc((size_t)m.Z * 4, s);
    c.val.alloc((size_t)m.Z * 4, s);
    to_coo(m, c.row.as<int32_t>(), c.col.as<int32_t>(), c.val.as<float>(), s);
    return csr_from_canon(std::move(c), s);
}

}  // namespace gs
