// Host-only arithmetic of the library, free of HIP so that it can also be
// built and checked on its own (sanitizer builds):
//   * the format predictor's model file, its normalisation and its tree
//     walk (Sec. 4.1, Sec. 4.4);
//   * the features of Table 2 (Sec. 4.4) as doubles from the exact integer
//     aggregates the device computes.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/gnnspmm.h"

namespace gs {

// Predictor inputs: F1..F19 of Table 2, the fill of 16x16 blocks
// (nnz / (256 n_blocks16)) and the width F of X.
constexpr int kNFeat = 21;

// The built-in model text (hand-set trees, model file version 1).
extern const char *const kBuiltinModel;

struct Node {
    int feat;
    double thr;
    int left, right;
    double value;
};
struct Tree {
    int cls;
    std::vector<Node> nodes;
};
struct Model {
    int k = 0;
    int cls_fmt[GS_NUM_FORMATS] = {0};
    double mn[kNFeat] = {0}, mx[kNFeat] = {0};
    double base[GS_NUM_FORMATS] = {0};
    std::vector<Tree> trees;
    double w = 1.0;  // the weight of Eq. 1 the model was trained for
};


// Parses a model file (versions 1 and 2, see gs_model.cpp).  On a malformed
// text returns false with *err set and m unchanged.
bool parse_model(const std::string &text, Model &m, std::string *err);

// Model input vector x[kNFeat] of a matrix with features f, for width F.
void model_input(const gs_features &f, int64_t F, double *x);

// Min-max scaling with the model's training range, clipped to [0, 1].
void normalise(const Model &m, double *x);

// Per-class scores: base plus the leaf value of every tree of the class.
void score(const Model &m, const double *x, double *sc);

// Population standard deviation sqrt((n S2 - Z^2) / n^2) of n counts with
// sum Z and sum of squares S2, the numerator formed exactly.
double population_dev(int64_t n, int64_t Z, uint64_t s2);

// The features of Table 2 from the integer aggregates already in f (n_rows,
// n_cols, nnz, n_diags, max/min row and column counts, sums of squared
// counts, bounces, n_blocks16): fills f->f[0..18] in Table 2 order.
void finish_features(gs_features *f);

}  // namespace gs
