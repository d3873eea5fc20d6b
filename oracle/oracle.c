/*
 * oracle.c -- plain, slow, obviously-correct CPU reference for the GNN
 * aggregation SpMM and everything around it.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The GPU library shares
 * no code, header, table or helper with this file and never calls it.
 *
 * What it computes, and where the paper defines it
 * ("Optimizing Sparse Matrix Multiplications for Graph Neural Networks",
 *  Qiu, You, Wang, arXiv 2111.00352):
 *
 *   - COO, CSR, DIA, BSR storage formats ............ Sec. 2.2
 *     ELL (row-packed, padded) is not in Sec. 2.2; it is the padded
 *     "packed structure" idea that Table 2 (feature F14) refers to.
 *   - SpMM Y = A.X, A the sparse adjacency, X dense .. Sec. 2.1
 *   - Matrix features F1..F19 ........................ Sec. 4.4, Table 2
 *     (the paper names the features but prints no formulas; the exact
 *      formulas below are this project's reading, stated per function).
 *
 * Canonical layouts (exactly one correct output per input):
 *   COO : triplets sorted by (row, col); no duplicates; no stored zeros.
 *   CSR : row_ptr[i] = #entries with row < i; col/val in canonical order.
 *   ELL : K = max row length; slot (i,k) at k*R+i (column-major); unused
 *         slots hold col = -1, val = +0.0f.
 *   DIA : offsets = ascending distinct (col-row); data[d*R+i] = A[i,i+off_d]
 *         or +0.0f (row-indexed, every diagonal padded to length R).
 *   BSR : block size b; blocks = distinct (row/b, col/b) ordered by block
 *         row then block column; block_val[blk*b*b + (row%b)*b + col%b];
 *         all other slots +0.0f.
 *
 * Every routine is a direct loop over the definition.  No blocking, no
 * fusion, no reordering beyond what the definition states.  Sums in the
 * SpMM are taken in fp64 in canonical column order.
 *
 * Parity status: SpMM, conversions and features are pinned by the tests in
 * tests/test_oracle_*.py (hand-worked example, dense brute force, closed
 * forms of GCN normalisation and of the 2-D grid, identity special cases,
 * round trips, and an independent numpy count of every integer aggregate).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Error codes, same numeric meaning as the GPU library's (both follow the
 * reading that explicit zeros and duplicates are rejected). */
#define OR_OK 0
#define OR_ERR_ARG (-1)
#define OR_ERR_INDEX (-2)
#define OR_ERR_DUPLICATE (-3)
#define OR_ERR_EXPLICIT_ZERO (-4)
#define OR_ERR_OOM (-6)

typedef struct {
    int32_t r, c;
    float v;
} or_trip;

static int cmp_trip(const void *pa, const void *pb)
{
    const or_trip *a = (const or_trip *)pa, *b = (const or_trip *)pb;
    if (a->r != b->r) return a->r < b->r ? -1 : 1;
    if (a->c != b->c) return a->c < b->c ? -1 : 1;
    return 0;
}

/* Canonical COO (Sec. 2.2, COO).  Checks, in this order of precedence:
 * index range (OR_ERR_INDEX), stored zeros (OR_ERR_EXPLICIT_ZERO),
 * duplicate coordinates (OR_ERR_DUPLICATE).  Then sorts by (row, col). */
int or_canon(int64_t R, int64_t C, int64_t Z, const int32_t *row, const int32_t *col,
             const float *val, int32_t *orow, int32_t *ocol, float *oval)
{
    if (R < 0 || C < 0 || Z < 0) return OR_ERR_ARG;
    for (int64_t k = 0; k < Z; k++)
        if (row[k] < 0 || row[k] >= R || col[k] < 0 || col[k] >= C) return OR_ERR_INDEX;
    for (int64_t k = 0; k < Z; k++)
        if (val[k] == 0.0f) return OR_ERR_EXPLICIT_ZERO;
    or_trip *t = (or_trip *)malloc((size_t)(Z > 0 ? Z : 1) * sizeof(or_trip));
    if (!t) return OR_ERR_OOM;
    for (int64_t k = 0; k < Z; k++) {
        t[k].r = row[k];
        t[k].c = col[k];
        t[k].v = val[k];
    }
    qsort(t, (size_t)Z, sizeof(or_trip), cmp_trip);
    for (int64_t k = 1; k < Z; k++)
        if (t[k].r == t[k - 1].r && t[k].c == t[k - 1].c) {
            free(t);
            return OR_ERR_DUPLICATE;
        }
    for (int64_t k = 0; k < Z; k++) {
        orow[k] = t[k].r;
        ocol[k] = t[k].c;
        oval[k] = t[k].v;
    }
    free(t);
    return OR_OK;
}

/* CSR row pointers from canonical COO rows (Sec. 2.2, CSR):
 * row_ptr[i] = number of entries whose row is < i. */
int or_csr(int64_t R, int64_t Z, const int32_t *crow, int32_t *row_ptr)
{
    for (int64_t i = 0; i <= R; i++) row_ptr[i] = 0;
    for (int64_t k = 0; k < Z; k++) row_ptr[crow[k] + 1] += 1;
    for (int64_t i = 0; i < R; i++) row_ptr[i + 1] += row_ptr[i];
    return OR_OK;
}

/* K of ELL: the longest row (0 for an empty matrix). */
int64_t or_ell_width(int64_t R, const int32_t *row_ptr)
{
    int64_t K = 0;
    for (int64_t i = 0; i < R; i++)
        if (row_ptr[i + 1] - row_ptr[i] > K) K = row_ptr[i + 1] - row_ptr[i];
    return K;
}

/* ELL fill: slot (i,k) at k*R+i holds the k-th entry of row i in column
 * order; padding is col = -1, val = +0.0f. */
int or_ell(int64_t R, int64_t K, const int32_t *row_ptr, const int32_t *col, const float *val,
           int32_t *ell_col, float *ell_val)
{
    for (int64_t k = 0; k < K; k++)
        for (int64_t i = 0; i < R; i++) {
            int64_t n = row_ptr[i + 1] - row_ptr[i];
            if (k < n) {
                ell_col[k * R + i] = col[row_ptr[i] + k];
                ell_val[k * R + i] = val[row_ptr[i] + k];
            } else {
                ell_col[k * R + i] = -1;
                ell_val[k * R + i] = 0.0f;
            }
        }
    return OR_OK;
}

/* ELL -> canonical COO: every slot with col != -1, rows in order, slots in
 * order within a row (which is column order).  Returns the count. */
int64_t or_ell_to_coo(int64_t R, int64_t K, const int32_t *ell_col, const float *ell_val,
                      int32_t *orow, int32_t *ocol, float *oval)
{
    int64_t z = 0;
    for (int64_t i = 0; i < R; i++)
        for (int64_t k = 0; k < K; k++)
            if (ell_col[k * R + i] != -1) {
                orow[z] = (int32_t)i;
                ocol[z] = ell_col[k * R + i];
                oval[z] = ell_val[k * R + i];
                z++;
            }
    return z;
}

/* DIA offsets (Sec. 2.2, DIA): the ascending distinct values of col-row.
 * Offsets range over [-(R-1), C-1].  Returns the number of diagonals. */
int64_t or_dia_offsets(int64_t R, int64_t C, int64_t Z, const int32_t *crow, const int32_t *ccol,
                       int32_t *offsets)
{
    if (R == 0 || C == 0) return 0;
    int64_t span = R + C - 1;
    unsigned char *seen = (unsigned char *)calloc((size_t)span, 1);
    if (!seen) return OR_ERR_OOM;
    for (int64_t k = 0; k < Z; k++) seen[(int64_t)ccol[k] - crow[k] + (R - 1)] = 1;
    int64_t nd = 0;
    for (int64_t s = 0; s < span; s++)
        if (seen[s]) {
            if (offsets) offsets[nd] = (int32_t)(s - (R - 1));
            nd++;
        }
    free(seen);
    return nd;
}

/* DIA fill: data[d*R+i] = A[i, i+offsets[d]] if stored, else +0.0f. */
int or_dia(int64_t R, int64_t ND, const int32_t *offsets, int64_t Z, const int32_t *crow,
           const int32_t *ccol, const float *cval, float *data)
{
    for (int64_t s = 0; s < ND * R; s++) data[s] = 0.0f;
    for (int64_t k = 0; k < Z; k++) {
        int32_t off = ccol[k] - crow[k];
        /* offsets are ascending: find off by binary search */
        int64_t lo = 0, hi = ND - 1;
        while (lo < hi) {
            int64_t mid = (lo + hi) / 2;
            if (offsets[mid] < off) lo = mid + 1;
            else hi = mid;
        }
        data[lo * R + crow[k]] = cval[k];
    }
    return OR_OK;
}

/* DIA -> canonical COO: per row, diagonals in ascending offset order give
 * ascending columns; a slot is an entry iff its value is nonzero and its
 * column lies inside [0, C). */
int64_t or_dia_to_coo(int64_t R, int64_t C, int64_t ND, const int32_t *offsets, const float *data,
                      int32_t *orow, int32_t *ocol, float *oval)
{
    int64_t z = 0;
    for (int64_t i = 0; i < R; i++)
        for (int64_t d = 0; d < ND; d++) {
            int64_t j = i + offsets[d];
            float v = data[d * R + i];
            if (j >= 0 && j < C && v != 0.0f) {
                orow[z] = (int32_t)i;
                ocol[z] = (int32_t)j;
                oval[z] = v;
                z++;
            }
        }
    return z;
}

/* BSR block structure (Sec. 2.2, BSR) for block size b: block_ptr over
 * ceil(R/b) block rows and the block columns, ascending per block row.
 * With block_col == NULL only counts.  Returns the number of blocks. */
int64_t or_bsr_structure(int64_t R, int64_t C, int64_t b, int64_t Z, const int32_t *crow,
                         const int32_t *ccol, int32_t *block_ptr, int32_t *block_col)
{
    if (b <= 0) return OR_ERR_ARG;
    int64_t nbr = (R + b - 1) / b, nbc = (C + b - 1) / b;
    unsigned char *mark = (unsigned char *)calloc((size_t)(nbc > 0 ? nbc : 1), 1);
    if (!mark) return OR_ERR_OOM;
    int64_t nb = 0;
    int64_t k = 0;
    for (int64_t br = 0; br < nbr; br++) {
        if (block_ptr) block_ptr[br] = (int32_t)nb;
        while (k < Z && crow[k] / b == br) {
            mark[ccol[k] / b] = 1;
            k++;
        }
        for (int64_t bc = 0; bc < nbc; bc++)
            if (mark[bc]) {
                if (block_col) block_col[nb] = (int32_t)bc;
                nb++;
                mark[bc] = 0;
            }
    }
    if (block_ptr) block_ptr[nbr] = (int32_t)nb;
    free(mark);
    return nb;
}

/* BSR values: block_val[blk*b*b + (row%b)*b + col%b]; all else +0.0f. */
int or_bsr_values(int64_t R, int64_t b, const int32_t *block_ptr, const int32_t *block_col,
                  int64_t nb, int64_t Z, const int32_t *crow, const int32_t *ccol, const float *cval,
                  float *block_val)
{
    (void)R;
    for (int64_t s = 0; s < nb * b * b; s++) block_val[s] = 0.0f;
    for (int64_t k = 0; k < Z; k++) {
        int64_t br = crow[k] / b, bc = ccol[k] / b;
        int64_t blk = block_ptr[br];
        while (block_col[blk] != bc) blk++; /* linear search in its block row */
        block_val[blk * b * b + (crow[k] % b) * b + (ccol[k] % b)] = cval[k];
    }
    return OR_OK;
}

/* BSR -> canonical COO: per row, blocks of its block row in ascending block
 * column, columns ascending inside a block; a slot is an entry iff nonzero
 * and inside the R x C matrix. */
int64_t or_bsr_to_coo(int64_t R, int64_t C, int64_t b, const int32_t *block_ptr,
                      const int32_t *block_col, const float *block_val, int32_t *orow,
                      int32_t *ocol, float *oval)
{
    int64_t z = 0;
    for (int64_t i = 0; i < R; i++) {
        int64_t br = i / b;
        for (int64_t blk = block_ptr[br]; blk < block_ptr[br + 1]; blk++)
            for (int64_t jj = 0; jj < b; jj++) {
                int64_t j = (int64_t)block_col[blk] * b + jj;
                float v = block_val[blk * b * b + (i % b) * b + jj];
                if (j < C && v != 0.0f) {
                    orow[z] = (int32_t)i;
                    ocol[z] = (int32_t)j;
                    oval[z] = v;
                    z++;
                }
            }
    }
    return z;
}

/* Matrix features, Sec. 4.4 / Table 2.  Integer aggregates first (exact),
 * then the 19 doubles in a fixed operation order.
 *
 *  ints[0..12] = R, C, Z, N_diags, max_r, min_r, max_c, min_c,
 *                sum r^2, sum c^2, sum |r_{i+1}-r_i|, sum |c_{j+1}-c_j|,
 *                number of distinct (row/16, col/16) blocks.
 *  f[0..18]    = F1 numRow, F2 numCol, F3 NNZ, F4 N_diags, F5 aver_RD,
 *                F6 max_RD, F7 min_RD, F8 dev_RD, F9 aver_CD, F10 max_CD,
 *                F11 min_CD, F12 dev_CD, F13 ER_DIA, F14 ER_CD,
 *                F15 row_bounce, F16 col_bounce, F17 density, F18 cv,
 *                F19 max_mu.
 *
 * Readings (the paper gives names and one-line descriptions only):
 *   dev     = population standard deviation, sqrt((n*S2 - Z^2)/n^2), with
 *             the numerator formed exactly in unsigned 128-bit arithmetic;
 *   ER_DIA  = Z / (N_diags * R)   (fill ratio of DIA storage);
 *   ER_CD   = Z / (C * max_CD)    (fill ratio of a column-packed layout);
 *   bounce  = mean |count difference| of adjacent rows (columns);
 *   cv      = dev_RD / aver_RD;  max_mu = max_RD - aver_RD;
 *   a ratio whose denominator is zero is 0. */
static double or_dev(int64_t n, int64_t Z, uint64_t s2)
{
    if (n == 0) return 0.0;
    unsigned __int128 a = (unsigned __int128)(uint64_t)n * s2;
    unsigned __int128 b = (unsigned __int128)(uint64_t)Z * (uint64_t)Z;
    unsigned __int128 num = a - b;
    double q = (double)num / ((double)n * (double)n);
    return sqrt(q);
}

int or_features(int64_t R, int64_t C, int64_t Z, const int32_t *crow, const int32_t *ccol,
                int64_t *ints, double *f)
{
    int64_t *rc = (int64_t *)calloc((size_t)(R > 0 ? R : 1), sizeof(int64_t));
    int64_t *cc = (int64_t *)calloc((size_t)(C > 0 ? C : 1), sizeof(int64_t));
    if (!rc || !cc) {
        free(rc);
        free(cc);
        return OR_ERR_OOM;
    }
    for (int64_t k = 0; k < Z; k++) {
        rc[crow[k]]++;
        cc[ccol[k]]++;
    }
    int64_t nd = or_dia_offsets(R, C, Z, crow, ccol, NULL);
    int64_t maxr = 0, minr = 0, maxc = 0, minc = 0;
    uint64_t s2r = 0, s2c = 0, br = 0, bc = 0;
    for (int64_t i = 0; i < R; i++) {
        if (i == 0 || rc[i] > maxr) maxr = rc[i];
        if (i == 0 || rc[i] < minr) minr = rc[i];
        s2r += (uint64_t)(rc[i] * rc[i]);
        if (i + 1 < R) br += (uint64_t)llabs(rc[i + 1] - rc[i]);
    }
    for (int64_t j = 0; j < C; j++) {
        if (j == 0 || cc[j] > maxc) maxc = cc[j];
        if (j == 0 || cc[j] < minc) minc = cc[j];
        s2c += (uint64_t)(cc[j] * cc[j]);
        if (j + 1 < C) bc += (uint64_t)llabs(cc[j + 1] - cc[j]);
    }
    int64_t nb16 = or_bsr_structure(R, C, 16, Z, crow, ccol, NULL, NULL);
    free(rc);
    free(cc);

    ints[0] = R; ints[1] = C; ints[2] = Z; ints[3] = nd;
    ints[4] = maxr; ints[5] = minr; ints[6] = maxc; ints[7] = minc;
    ints[8] = (int64_t)s2r; ints[9] = (int64_t)s2c;
    ints[10] = (int64_t)br; ints[11] = (int64_t)bc; ints[12] = nb16;

    double dR = (double)R, dC = (double)C, dZ = (double)Z;
    double aver_rd = R > 0 ? dZ / dR : 0.0;
    double aver_cd = C > 0 ? dZ / dC : 0.0;
    double dev_rd = or_dev(R, Z, s2r);
    double dev_cd = or_dev(C, Z, s2c);
    f[0] = dR;
    f[1] = dC;
    f[2] = dZ;
    f[3] = (double)nd;
    f[4] = aver_rd;
    f[5] = (double)maxr;
    f[6] = (double)minr;
    f[7] = dev_rd;
    f[8] = aver_cd;
    f[9] = (double)maxc;
    f[10] = (double)minc;
    f[11] = dev_cd;
    f[12] = (nd > 0 && R > 0) ? dZ / ((double)nd * dR) : 0.0;
    f[13] = (C > 0 && maxc > 0) ? dZ / (dC * (double)maxc) : 0.0;
    f[14] = R > 1 ? (double)br / (double)(R - 1) : 0.0;
    f[15] = C > 1 ? (double)bc / (double)(C - 1) : 0.0;
    f[16] = (R > 0 && C > 0) ? dZ / (dR * dC) : 0.0;
    f[17] = aver_rd != 0.0 ? dev_rd / aver_rd : 0.0;
    f[18] = (double)maxr - aver_rd;
    return OR_OK;
}

/* SpMM, Sec. 2.1: Y[i,f] = sum over the entries (i,j,a) of row i, in column
 * order, of a * X[j,f], accumulated in fp64.  M[i,f] = sum |a| * |X[j,f]|
 * (the scale of the tolerance bound).  Rows are independent; each row is
 * summed by one thread in a fixed order, so the result does not depend on
 * the thread count. */
int or_spmm(int64_t R, const int32_t *row_ptr, const int32_t *col, const float *val,
            const float *X, int64_t ldx, int64_t F, double *Y, double *M)
{
    int64_t i;
#pragma omp parallel for schedule(dynamic, 64)
    for (i = 0; i < R; i++) {
        for (int64_t f = 0; f < F; f++) {
            double s = 0.0, m = 0.0;
            for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; k++) {
                double a = (double)val[k];
                double x = (double)X[(int64_t)col[k] * ldx + f];
                s += a * x;
                m += fabs(a) * fabs(x);
            }
            Y[i * F + f] = s;
            if (M) M[i * F + f] = m;
        }
    }
    return OR_OK;
}

/* The same sum with an fp64 dense operand (Sec. 2.1): used where the dense
 * input is itself an exact fp64 intermediate (a GNN layer's hidden features
 * or gradients), so that nothing is rounded to fp32 along a layer chain. */
int or_spmm64(int64_t R, const int32_t *row_ptr, const int32_t *col, const float *val,
              const double *X, int64_t ldx, int64_t F, double *Y)
{
    int64_t i;
#pragma omp parallel for schedule(dynamic, 64)
    for (i = 0; i < R; i++) {
        for (int64_t f = 0; f < F; f++) {
            double s = 0.0;
            for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; k++)
                s += (double)val[k] * X[(int64_t)col[k] * ldx + f];
            Y[i * F + f] = s;
        }
    }
    return OR_OK;
}

/* Same definition, for a chosen list of rows only (used to check sampled
 * outputs of very large problems one row at a time). */
int or_spmm_rows(int64_t nsel, const int64_t *rows, const int32_t *row_ptr, const int32_t *col,
                 const float *val, const float *X, int64_t ldx, int64_t F, double *Y, double *M)
{
    for (int64_t s = 0; s < nsel; s++) {
        int64_t i = rows[s];
        for (int64_t f = 0; f < F; f++) {
            double acc = 0.0, m = 0.0;
            for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; k++) {
                double a = (double)val[k];
                double x = (double)X[(int64_t)col[k] * ldx + f];
                acc += a * x;
                m += fabs(a) * fabs(x);
            }
            Y[s * F + f] = acc;
            if (M) M[s * F + f] = m;
        }
    }
    return OR_OK;
}

int or_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of later parallel loops (timing only; results do not depend on it:
 * every row is summed by one thread in one fixed order). */
void or_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
