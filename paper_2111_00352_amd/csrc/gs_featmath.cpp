// The features of Table 2 (Sec. 4.4) as doubles, from the exact integer
// aggregates the device computes (host only).  Every operation is IEEE
// round-to-nearest in the order written, so the doubles are reproducible:
//   dev = sqrt((n S2 - Z^2) / (n n)) with the numerator exact,
//   ER_DIA = Z / (N_diags R), ER_CD = Z / (C max_CD),
//   bounce = sum |count difference of adjacent rows (columns)| / (R-1) (C-1),
//   density = Z / (R C), cv = dev_RD / aver_RD, max_mu = max_RD - aver_RD;
// a ratio whose denominator is zero is 0.
#include <cmath>

#include "gs_host.h"

namespace gs {

// n S2 - Z^2 >= 0 (Cauchy-Schwarz), formed exactly in 128-bit arithmetic.
double population_dev(int64_t n, int64_t Z, uint64_t s2)
{
    if (n <= 0) return 0.0;
    const unsigned __int128 num = (unsigned __int128)(uint64_t)n * s2 -
                                  (unsigned __int128)(uint64_t)Z * (uint64_t)Z;
    const double q = (double)num / ((double)n * (double)n);
    return std::sqrt(q);
}

void finish_features(gs_features *out)
{
    gs_features &f = *out;
    const int64_t R = f.n_rows, C = f.n_cols, Z = f.nnz;
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
