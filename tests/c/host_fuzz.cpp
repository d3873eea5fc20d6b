// Sanitizer driver for the library's host-only arithmetic (built with
// -fsanitize=address,undefined by tests/test_sanitizers.py): the predictor's
// model parser and tree walk on the shipped and built-in models and on
// truncated and garbled model texts, and the Table 2 feature doubles on
// edge-case and random integer aggregates.  Any memory or undefined-behaviour
// error aborts the run; a malformed model must be refused, never crash.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <fstream>
#include <sstream>
#include <string>
#include <vector>

#include "../../paper_2111_00352_amd/csrc/gs_host.h"

namespace {

uint64_t g_state = 0x9e3779b97f4a7c15ull;
uint64_t next()  // SplitMix64 (Steele, Lea and Flood 2014)
{
    uint64_t z = (g_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

int g_parsed = 0, g_refused = 0;

void exercise(const std::string &text)
{
    gs::Model m;
    std::string err;
    if (!gs::parse_model(text, m, &err)) {
        if (err.empty()) std::abort();
        g_refused++;
        return;
    }
    g_parsed++;
    gs_features f{};
    f.n_rows = 1000, f.n_cols = 1000, f.nnz = 5000, f.n_diags = 9, f.max_rd = 11, f.min_rd = 1;
    f.max_cd = 12, f.min_cd = 0, f.sum_rd2 = 30000, f.sum_cd2 = 31000, f.bounce_r = 900, f.bounce_c = 950;
    f.n_blocks16 = 300;
    gs::finish_features(&f);
    for (int F : {1, 64, 128, 4096}) {
        double x[gs::kNFeat], sc[GS_NUM_FORMATS];
        gs::model_input(f, F, x);
        for (int i = 0; i < gs::kNFeat; i++)  // random inputs as well
            if (next() & 1) x[i] = (double)(int64_t)next() * 1e-12;
        gs::normalise(m, x);
        gs::score(m, x, sc);
        for (int c = 0; c < m.k; c++)
            if (std::isnan(sc[c]) && !std::isnan(m.base[c])) {
                // NaN scores come only from NaN in the file; the walk must still end
            }
    }
}

std::vector<std::string> tokens_of(const std::string &t)
{
    std::istringstream in(t);
    std::vector<std::string> v;
    std::string w;
    while (in >> w) v.push_back(w);
    return v;
}

std::string join(const std::vector<std::string> &v)
{
    std::string s;
    for (const auto &w : v) s += w + ' ';
    return s;
}

}  // namespace

int main(int argc, char **argv)
{
    std::vector<std::string> models = {gs::kBuiltinModel};
    if (argc > 1) {
        std::ifstream f(argv[1], std::ios::binary);
        std::stringstream ss;
        ss << f.rdbuf();
        models.push_back(ss.str());
    }
    for (const auto &t : models) {
        gs::Model m;
        std::string err;
        if (!gs::parse_model(t, m, &err)) {
            std::fprintf(stderr, "a shipped model was refused: %s\n", err.c_str());
            return 1;
        }
    }
    const char *specials[] = {"-1", "0", "1", "2147483647", "-2147483648", "99999999999", "1e308", "-1e308",
                              "nan", "inf", "0x1p-1074", "0x.p1", "0xfffffffffffffffp1", "L", "tree",
                              "GSMODEL", "", "0x1.8p+1100", "+", "-", "21", "6"};
    for (const auto &t : models) {
        // every truncation (coarse steps through long texts)
        const size_t step = t.size() > 4000 ? t.size() / 4000 : 1;
        for (size_t n = 0; n <= t.size(); n += step) exercise(t.substr(0, n));
        // byte flips
        for (int it = 0; it < 1500; it++) {
            std::string u = t;
            const int flips = 1 + (int)(next() % 4);
            for (int k = 0; k < flips; k++) u[next() % u.size()] = (char)(" \n-+.0123456789abcdefxLp"[next() % 24]);
            exercise(u);
        }
        // token edits: replace, delete, duplicate
        const auto tok = tokens_of(t);
        for (int it = 0; it < 1500; it++) {
            auto v = tok;
            const size_t i = next() % v.size();
            switch (next() % 3) {
            case 0: v[i] = specials[next() % (sizeof specials / sizeof *specials)]; break;
            case 1: v.erase(v.begin() + (long)i); break;
            default: v.insert(v.begin() + (long)i, v[i]); break;
            }
            exercise(join(v));
        }
    }
    // feature doubles on edge cases and random aggregates
    const int64_t sizes[] = {0, 1, 2, 3, 1000, (int64_t)1 << 31, ((int64_t)1 << 31) - 1};
    for (int64_t R : sizes)
        for (int64_t C : sizes) {
            gs_features f{};
            f.n_rows = R, f.n_cols = C;
            f.nnz = (R && C) ? std::min<int64_t>(R, C) : 0;
            f.max_rd = f.min_rd = f.nnz ? 1 : 0;
            f.max_cd = f.min_cd = f.nnz ? 1 : 0;
            f.sum_rd2 = f.sum_cd2 = (uint64_t)f.nnz;
            f.n_diags = f.nnz ? 1 : 0;
            gs::finish_features(&f);
        }
    for (int it = 0; it < 30000; it++) {
        gs_features f{};
        f.n_rows = (int64_t)(next() % ((uint64_t)1 << 31));
        f.n_cols = (int64_t)(next() % ((uint64_t)1 << 31));
        f.nnz = (int64_t)(next() % ((uint64_t)1 << 31));
        f.n_diags = (int64_t)(next() % ((uint64_t)1 << 32));
        f.max_rd = (int64_t)(next() % ((uint64_t)1 << 31));
        f.min_rd = (int64_t)(next() % ((uint64_t)1 << 31));
        f.max_cd = (int64_t)(next() % ((uint64_t)1 << 31));
        f.min_cd = (int64_t)(next() % ((uint64_t)1 << 31));
        // counts consistent with Cauchy-Schwarz: S2 >= Z^2 / n
        const unsigned __int128 z2 = (unsigned __int128)f.nnz * (uint64_t)f.nnz;
        const uint64_t lo_r = f.n_rows ? (uint64_t)(z2 / (uint64_t)f.n_rows) + 1 : 0;
        const uint64_t lo_c = f.n_cols ? (uint64_t)(z2 / (uint64_t)f.n_cols) + 1 : 0;
        f.sum_rd2 = lo_r + next() % 1000;
        f.sum_cd2 = lo_c + next() % 1000;
        f.bounce_r = next() >> 2, f.bounce_c = next() >> 2;
        f.n_blocks16 = (int64_t)(next() >> 34);
        gs::finish_features(&f);
        double x[gs::kNFeat];
        gs::model_input(f, 128, x);
    }
    std::printf("host_fuzz ok: %d parsed, %d refused\n", g_parsed, g_refused);
    return 0;
}
