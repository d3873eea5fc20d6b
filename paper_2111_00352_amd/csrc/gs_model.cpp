// The format predictor's model file and tree walk (host only).
//
// Model file (text, whitespace separated):
//   GSMODEL 1
//   nfeat <n>                       n = 21: F1..F19 of Table 2, then
//                                   bsr16_fill = nnz / (256 * n_blocks16)
//                                   and F (the width of X)
//   classes <k> <format id> x k     class index -> gs_format
//   min <n doubles>   max <n doubles>
//   base <k doubles>                initial score of each class
//   ntrees <T>
//   T times:  tree <class> <nnodes>
//             nnodes lines: <feat> <threshold> <left> <right> <value>
//             (feat -1 = leaf with score value; otherwise x[feat] < threshold
//              goes to left, else right; node 0 is the root)
// Version 2 writes every real as a hexadecimal literal and leaves as
// "L value", internal nodes as "feat thr left right".
#include <cctype>
#include <climits>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <new>

#include "gs_host.h"

namespace gs {

// Built-in model: hand-set score trees standing in for a trained ensemble.
// Features are scaled by the given ranges; thresholds are in scaled units.
// CSR is the default (base score 1); DIA wins when nearly all stored slots
// of few diagonals are filled (ER_DIA >= 0.6, at most 64 diagonals), ELL when
// rows are near-uniform (cv < 0.05) and short (max_RD < 64), BSR when 16x16
// blocks are mostly full (fill >= 0.5).  These thresholds restate what the
// per-format SpMM timings on MI355X show; a trained ensemble in the same
// file format replaces them through model_path.
const char *const kBuiltinModel = R"(GSMODEL 1
nfeat 21
classes 5 1 0 2 3 4
min 0 0 0 0 0 0 0 0 0 0 0 0 0 0 0 0 0 0 0 0 0
max 1e8 1e8 1e10 1e7 1e4 1e5 1e4 1e4 1e4 1e5 1e4 1e4 1 1 1e4 1e4 1 100 1e5 1 4096
base 1 0.5 0 0 0
ntrees 3
tree 3 5
12 0.6 1 2 0
-1 0 0 0 -10
3 6.4e-6 3 4 0
-1 0 0 0 2
-1 0 0 0 -10
tree 2 5
17 0.0005 1 2 0
5 6.4e-4 3 4 0
-1 0 0 0 -5
-1 0 0 0 1.5
-1 0 0 0 -5
tree 4 3
19 0.5 1 2 0
-1 0 0 0 -10
-1 0 0 0 2.5
)";

namespace {

// Whitespace-separated tokens of the model text.  Numbers are read with
// strtod / strtol (the conversions the C library defines; a double rounds
// correctly) and must fill their whole token.
struct Tokens {
    const char *p;
    static bool space(char c) { return c == ' ' || c == '\n' || c == '\t' || c == '\r' || c == '\v' || c == '\f'; }
    bool word(const char *&s, const char *&e)
    {
        while (*p && space(*p)) p++;
        if (!*p) return false;
        s = p;
        while (*p && !space(*p)) p++;
        e = p;
        return true;
    }
    bool is(const char *w)
    {
        const char *s, *e;
        return word(s, e) && (size_t)(e - s) == std::strlen(w) && std::strncmp(s, w, e - s) == 0;
    }
    bool num(double &v)
    {
        const char *s, *e;
        if (!word(s, e)) return false;
        char *q = nullptr;
        v = std::strtod(s, &q);
        return q == e;
    }
    // A hexadecimal floating-point literal as C99 and Python's float.hex()
    // write it, [-]0xH.HHHp[+-]E: exact by construction, so it is read
    // without a general decimal conversion.  At most 53 significant bits.
    bool hexnum(double &v)
    {
        const char *s, *e;
        if (!word(s, e)) return false;
        const char *p = s;
        const bool neg = *p == '-';
        if (*p == '-' || *p == '+') p++;
        if (e - p < 4 || p[0] != '0' || (p[1] != 'x' && p[1] != 'X')) return false;
        p += 2;
        uint64_t m = 0;
        int frac = 0, nd = 0;
        bool dot = false;
        for (; p < e && *p != 'p' && *p != 'P'; p++) {
            if (*p == '.') {
                if (dot) return false;
                dot = true;
                continue;
            }
            const int d = std::isdigit((unsigned char)*p) ? *p - '0'
                          : (*p >= 'a' && *p <= 'f') ? *p - 'a' + 10
                          : (*p >= 'A' && *p <= 'F') ? *p - 'A' + 10
                                                     : -1;
            if (d < 0 || nd == 15) return false;
            m = m * 16 + (uint64_t)d;
            nd++;
            if (dot) frac++;
        }
        long long ex;
        if (nd == 0 || p == e || (m >> 53) != 0 || !integer(p + 1, e, -1100, 1100, ex)) return false;
        v = std::ldexp((double)m, (int)(ex - 4 * frac));
        if (neg) v = -v;
        return true;
    }
    // A decimal integer filling [s, e), within the int range.
    static bool integer(const char *s, const char *e, long long lo, long long hi, long long &x)
    {
        const bool neg = s < e && *s == '-';
        if (s < e && (*s == '-' || *s == '+')) s++;
        if (s == e || e - s > 11) return false;
        x = 0;
        for (; s < e; s++) {
            if (*s < '0' || *s > '9') return false;
            x = x * 10 + (*s - '0');
        }
        if (neg) x = -x;
        return x >= lo && x <= hi;
    }
    bool num(int &v)
    {
        const char *s, *e;
        long long x;
        if (!word(s, e) || !integer(s, e, INT_MIN, INT_MAX, x)) return false;
        v = (int)x;
        return true;
    }
};

// Model file, version 1: "GSMODEL 1", "nfeat 21", "classes k id...",
// "min x...", "max x...", "base s...", "ntrees N", then per tree
// "tree cls nn" and nn nodes "feat thr left right value" (feat = -1 for a
// leaf), numbers in decimal.  Version 2 is the same with every real written
// as a hexadecimal literal and leaves as "L value", internal nodes as
// "feat thr left right".  Either may end with "w x": the weight of Eq. 1
// whose labels the model learned (1 when absent).
struct ModelError {
    std::string msg;
};

[[noreturn]] void bad(const std::string &msg) { throw ModelError{"model: " + msg}; }

void parse(const std::string &text, Model &m)
{
    Tokens in{text.c_str()};
    int ver = 0, nf = 0;
    // every node takes at least two bytes of text: a longer list is a
    // malformed count, not a reason to reserve its memory
    const long long cap = (long long)text.size() / 2 + 1;
    auto expect = [&](const char *w) {
        if (!in.is(w)) bad(std::string("expected '") + w + "'");
    };
    expect("GSMODEL");
    if (!in.num(ver) || (ver != 1 && ver != 2)) bad("unsupported version");
    auto real = [&](double &v) { return ver == 1 ? in.num(v) : in.hexnum(v); };
    expect("nfeat");
    if (!in.num(nf) || nf != kNFeat) bad("nfeat must be " + std::to_string(kNFeat));
    expect("classes");
    if (!in.num(m.k) || m.k < 1 || m.k > GS_NUM_FORMATS) bad("bad class count");
    for (int c = 0; c < m.k; c++)
        if (!in.num(m.cls_fmt[c]) || m.cls_fmt[c] < 0 || m.cls_fmt[c] >= GS_NUM_FORMATS)
            bad("bad class format id");
    expect("min");
    for (int i = 0; i < kNFeat; i++)
        if (!real(m.mn[i])) bad("short min table");
    expect("max");
    for (int i = 0; i < kNFeat; i++)
        if (!real(m.mx[i])) bad("short max table");
    expect("base");
    for (int c = 0; c < m.k; c++)
        if (!real(m.base[c])) bad("short base scores");
    int nt = 0;
    expect("ntrees");
    if (!in.num(nt) || nt < 0 || nt > cap) bad("bad tree count");
    m.trees.resize(nt);
    for (auto &t : m.trees) {
        int nn = 0;
        expect("tree");
        if (!in.num(t.cls) || !in.num(nn) || t.cls < 0 || t.cls >= m.k || nn < 1 || nn > cap)
            bad("bad tree header");
        t.nodes.resize(nn);
        for (auto &n : t.nodes) {
            bool ok;
            if (ver == 1) {
                ok = in.num(n.feat) && in.num(n.thr) && in.num(n.left) && in.num(n.right) && in.num(n.value);
            } else {
                const char *save = in.p;
                if (in.is("L")) {
                    n = Node{-1, 0.0, 0, 0, 0.0};
                    ok = in.hexnum(n.value);
                } else {
                    in.p = save;
                    n.value = 0.0;
                    ok = in.num(n.feat) && n.feat >= 0 && in.hexnum(n.thr) && in.num(n.left) && in.num(n.right);
                }
            }
            if (!ok) bad("short or malformed node list");
        }
        for (int i = 0; i < nn; i++) {
            const Node &n = t.nodes[i];
            if (n.feat >= kNFeat || n.feat < -1) bad("bad feature index");
            if (n.feat >= 0 && (n.left <= i || n.right <= i || n.left >= nn || n.right >= nn))
                bad("bad child index");
        }
    }
    const char *save = in.p;
    if (in.is("w")) {
        if (!real(m.w) || !(m.w >= 0.0 && m.w <= 1.0)) bad("w must be in [0, 1]");
    } else {
        in.p = save;
    }
}

}  // namespace

bool parse_model(const std::string &text, Model &m, std::string *err)
{
    Model fresh;
    try {
        parse(text, fresh);
    } catch (const ModelError &e) {
        if (err) *err = e.msg;
        return false;
    } catch (const std::bad_alloc &) {
        if (err) *err = "model: out of host memory";
        return false;
    }
    m = std::move(fresh);
    return true;
}

// Model input: F1..F19, the fill of 16x16 blocks, and the width F of X.
void model_input(const gs_features &f, int64_t F, double *x)
{
    for (int i = 0; i < 19; i++) x[i] = f.f[i];
    x[19] = f.n_blocks16 > 0 ? (double)f.nnz / (256.0 * (double)f.n_blocks16) : 0.0;
    x[20] = (double)F;
}

// Min-max scaling to [0,1] with the training range, clipped (Sec. 4.4), then
// rounded to fp32: tree thresholds are learned on fp32 features.
void normalise(const Model &m, double *x)
{
    for (int i = 0; i < kNFeat; i++) {
        const double span = m.mx[i] - m.mn[i];
        double v = span > 0 ? (x[i] - m.mn[i]) / span : 0.0;
        v = v < 0 ? 0 : (v > 1 ? 1 : v);
        x[i] = (double)(float)v;
    }
}

void score(const Model &m, const double *x, double *sc)
{
    for (int c = 0; c < m.k; c++) sc[c] = m.base[c];
    for (const auto &t : m.trees) {
        int i = 0;
        while (t.nodes[i].feat >= 0) i = x[t.nodes[i].feat] < t.nodes[i].thr ? t.nodes[i].left : t.nodes[i].right;
        sc[t.cls] += t.nodes[i].value;
    }
}


}  // namespace gs
