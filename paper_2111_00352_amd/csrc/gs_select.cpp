// Per-layer format selection and dispatch (Sec. 4, Sec. 4.6): features are
// extracted once per adjacency key (Sec. 4.4), min-max normalised and
// clipped with the model's training range, scored by a boosted tree
// ensemble (Sec. 4.1; one score per candidate format, highest wins), the
// matrix is converted only when the chosen format has not been built for
// this key yet, and the chosen format's kernel runs.
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
#include <cctype>
#include <cerrno>
#include <chrono>
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <unordered_map>
#include <vector>

#include "gs_internal.h"

namespace gs {
gs_matrix_ *build_csr(const gs_coo *A, const gs_build_opts &o, hipStream_t s, bool plan);
void check_coo(const gs_coo *A);
}  // namespace gs

using namespace gs;

namespace {

constexpr int kNFeat = 21;

// Built-in model: hand-set score trees standing in for a trained ensemble.
// Features are scaled by the given ranges; thresholds are in scaled units.
// CSR is the default (base score 1); DIA wins when nearly all stored slots
// of few diagonals are filled (ER_DIA >= 0.6, at most 64 diagonals), ELL when
// rows are near-uniform (cv < 0.05) and short (max_RD < 64), BSR when 16x16
// blocks are mostly full (fill >= 0.5).  These thresholds restate what the
// per-format SpMM timings on MI355X show; a trained ensemble in the same
// file format replaces them through model_path.
const char *kBuiltinModel = R"(GSMODEL 1
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
};

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
// "feat thr left right".
void parse_model(const std::string &text, Model &m)
{
    Tokens in{text.c_str()};
    int ver = 0, nf = 0;
    auto expect = [&](const char *w) {
        if (!in.is(w)) fail(GS_ERR_MODEL, "model: expected '%s'", w);
    };
    expect("GSMODEL");
    if (!in.num(ver) || (ver != 1 && ver != 2)) fail(GS_ERR_MODEL, "model: unsupported version");
    auto real = [&](double &v) { return ver == 1 ? in.num(v) : in.hexnum(v); };
    expect("nfeat");
    if (!in.num(nf) || nf != kNFeat) fail(GS_ERR_MODEL, "model: nfeat must be %d", kNFeat);
    expect("classes");
    if (!in.num(m.k) || m.k < 1 || m.k > GS_NUM_FORMATS) fail(GS_ERR_MODEL, "model: bad class count");
    for (int c = 0; c < m.k; c++)
        if (!in.num(m.cls_fmt[c]) || m.cls_fmt[c] < 0 || m.cls_fmt[c] >= GS_NUM_FORMATS)
            fail(GS_ERR_MODEL, "model: bad class format id");
    expect("min");
    for (int i = 0; i < kNFeat; i++)
        if (!real(m.mn[i])) fail(GS_ERR_MODEL, "model: short min table");
    expect("max");
    for (int i = 0; i < kNFeat; i++)
        if (!real(m.mx[i])) fail(GS_ERR_MODEL, "model: short max table");
    expect("base");
    for (int c = 0; c < m.k; c++)
        if (!real(m.base[c])) fail(GS_ERR_MODEL, "model: short base scores");
    int nt = 0;
    expect("ntrees");
    if (!in.num(nt) || nt < 0) fail(GS_ERR_MODEL, "model: bad tree count");
    m.trees.resize(nt);
    for (auto &t : m.trees) {
        int nn = 0;
        expect("tree");
        if (!in.num(t.cls) || !in.num(nn) || t.cls < 0 || t.cls >= m.k || nn < 1)
            fail(GS_ERR_MODEL, "model: bad tree header");
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
            if (!ok) fail(GS_ERR_MODEL, "model: short or malformed node list");
        }
        for (int i = 0; i < nn; i++) {
            const Node &n = t.nodes[i];
            if (n.feat >= kNFeat || n.feat < -1) fail(GS_ERR_MODEL, "model: bad feature index");
            if (n.feat >= 0 && (n.left <= i || n.right <= i || n.left >= nn || n.right >= nn))
                fail(GS_ERR_MODEL, "model: bad child index");
        }
    }
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

// Tie order when scores or times are equal.
constexpr int kTieOrder[GS_NUM_FORMATS] = {GS_CSR, GS_COO, GS_ELL, GS_DIA, GS_BSR, GS_CSC};

double now_s()
{
    return std::chrono::duration<double>(std::chrono::steady_clock::now().time_since_epoch()).count();
}

struct Entry {
    gs_features feat{};
    gs_matrix_ *built[GS_NUM_FORMATS] = {};
    uint64_t bytes[GS_NUM_FORMATS] = {0};
    int feasible = 0;
    std::unordered_map<int64_t, int> profiled;  // F -> fastest format
    struct Prediction {
        int fmt;
        double scores[GS_NUM_FORMATS];
    };
    std::unordered_map<int64_t, Prediction> predicted;  // F -> the model's choice
    double prof_time[GS_NUM_FORMATS] = {0};
    double t_features = 0, t_convert[GS_NUM_FORMATS] = {0};
    ~Entry()
    {
        for (auto *m : built) delete m;
    }
};

}  // namespace

struct gs_ctx_ {
    gs_selector_opts opts{};
    Model model;
    std::unordered_map<uint64_t, Entry *> cache;
    gs_select_stats last{};
    ~gs_ctx_()
    {
        for (auto &kv : cache) delete kv.second;
    }
};

namespace {

Entry &lookup(gs_ctx_ &c, uint64_t key, const gs_coo *A, hipStream_t s)
{
    auto it = c.cache.find(key);
    if (it != c.cache.end()) return *it->second;
    check_coo(A);
    Entry *e = new Entry();
    try {
        const double t0 = now_s();
        gs_build_opts o = {c.opts.bsr_block, 0, c.opts.max_bytes};
        gs_matrix_ *csr = build_csr(A, o, s, false);  // planned when CSR is first run
        e->built[GS_CSR] = csr;
        if (c.opts.mode == GS_SEL_FIXED) {
            // a fixed format needs no features: its build reports whether it fits
            e->feasible = (1 << GS_NUM_FORMATS) - 1;
            e->t_features = now_s() - t0;
            c.cache[key] = e;
            return *e;
        }
        features_from_csr(*csr, s, &e->feat);
        const int b = c.opts.bsr_block;
        const int64_t nb = (b == 16) ? e->feat.n_blocks16 : count_blocks(*csr, b, s);
        const gs_features &f = e->feat;
        for (int fmt = 0; fmt < GS_NUM_FORMATS; fmt++) {
            e->bytes[fmt] = format_bytes(fmt, f.n_rows, f.n_cols, f.nnz, f.max_rd, f.n_diags, nb, b);
            if (fmt == GS_CSR || fmt == GS_COO || fmt == GS_CSC || e->bytes[fmt] <= c.opts.max_bytes)
                e->feasible |= 1 << fmt;
        }
        e->t_features = now_s() - t0;
    } catch (...) {
        delete e;
        throw;
    }
    c.cache[key] = e;
    return *e;
}

gs_matrix_ &ensure_built(gs_ctx_ &c, Entry &e, int fmt, hipStream_t s)
{
    if (!e.built[fmt]) {
        const double t0 = now_s();
        e.built[fmt] = convert_from_csr(*e.built[GS_CSR], fmt, c.opts.bsr_block, c.opts.max_bytes, s,
                                        nullptr);
        e.t_convert[fmt] = now_s() - t0;
    } else if (fmt == GS_CSR && !e.built[fmt]->csr_planned) {
        const double t0 = now_s();
        plan_csr(*e.built[fmt], s);
        e.t_convert[fmt] = now_s() - t0;
    }
    return *e.built[fmt];
}

int choose(gs_ctx_ &c, Entry &e, int64_t F, const float *X, int64_t ldx, float *Y, int64_t ldy,
           hipStream_t s)
{
    gs_select_stats &st = c.last;
    st = gs_select_stats{};
    st.feasible_mask = e.feasible;
    st.t_features = e.t_features;
    int chosen = -1;
    const double t0 = now_s();
    if (c.opts.mode == GS_SEL_FIXED) {
        chosen = c.opts.fixed;
        if (!(e.feasible & (1 << chosen)))
            fail(GS_ERR_INFEASIBLE, "fixed format %d needs %llu bytes, over the cap", chosen,
                 (unsigned long long)e.bytes[chosen]);
    } else if (c.opts.mode == GS_SEL_MODEL) {
        // the inputs are the key's features and F, so the choice is made
        // once per (key, F) and reused on later calls (later epochs)
        auto it = e.predicted.find(F);
        if (it == e.predicted.end()) {
            Entry::Prediction p{};
            double x[kNFeat], sc[GS_NUM_FORMATS];
            model_input(e.feat, F, x);
            normalise(c.model, x);
            score(c.model, x, sc);
            double best = -1e300;
            int pick = -1;
            for (int fmt : kTieOrder) {
                if (!(e.feasible & c.opts.formats & (1u << fmt))) continue;
                for (int k = 0; k < c.model.k; k++)
                    if (c.model.cls_fmt[k] == fmt) {
                        p.scores[fmt] = sc[k];
                        if (sc[k] > best) {
                            best = sc[k];
                            pick = fmt;
                        }
                    }
            }
            p.fmt = pick < 0 ? GS_CSR : pick;  // the model scores no feasible format: CSR
            it = e.predicted.emplace(F, p).first;
        }
        chosen = it->second.fmt;
        for (int f = 0; f < GS_NUM_FORMATS; f++) st.scores[f] = it->second.scores[f];
    } else {  // GS_SEL_PROFILE: the exhaustive-search reference
        auto it = e.profiled.find(F);
        if (it != e.profiled.end()) {
            chosen = it->second;
        } else {
            if (!X || !Y) fail(GS_ERR_INVALID_ARG, "profiling needs X and Y");
            const int reps = c.opts.profile_reps > 0 ? c.opts.profile_reps : 3;
            hipEvent_t a, b;
            GS_HIP(hipEventCreate(&a));
            GS_HIP(hipEventCreate(&b));
            double best = 1e300;
            try {
                for (int fmt : kTieOrder) {
                    if (!(e.feasible & c.opts.formats & (1u << fmt))) continue;
                    gs_matrix_ &m = ensure_built(c, e, fmt, s);
                    run_spmm(m, X, ldx, Y, ldy, F, s);  // warm-up (and workspace growth)
                    GS_HIP(hipEventRecord(a, s));
                    for (int r = 0; r < reps; r++) run_spmm(m, X, ldx, Y, ldy, F, s);
                    GS_HIP(hipEventRecord(b, s));
                    GS_HIP(hipEventSynchronize(b));
                    float ms = 0;
                    GS_HIP(hipEventElapsedTime(&ms, a, b));
                    const double t = ms * 1e-3 / reps;
                    e.prof_time[fmt] = t;
                    if (t < best * 0.99) {  // within 1%: keep the earlier one in tie order
                        best = t;
                        chosen = fmt;
                    }
                }
            } catch (...) {
                (void)hipEventDestroy(a);
                (void)hipEventDestroy(b);
                throw;
            }
            (void)hipEventDestroy(a);
            (void)hipEventDestroy(b);
            if (chosen < 0) chosen = GS_CSR;  // no feasible candidate: the fallback
            e.profiled[F] = chosen;
        }
        for (int f = 0; f < GS_NUM_FORMATS; f++) st.scores[f] = e.prof_time[f];
    }
    st.t_predict = now_s() - t0;
    ensure_built(c, e, chosen, s);
    st.t_convert = e.t_convert[chosen];
    st.chosen = chosen;
    return chosen;
}

}  // namespace

extern "C" {

int gs_ctx_create(const gs_selector_opts *o, gs_ctx *out)
{
    if (out) *out = nullptr;
    return guarded([&] {
        if (!out) fail(GS_ERR_INVALID_ARG, "null output handle");
        gs_selector_opts r = {GS_SEL_MODEL, GS_CSR, nullptr, kDefaultMaxBytes, kDefaultBsrBlock, 3, 0};
        if (o) r = *o;
        constexpr uint32_t kAll = (1u << GS_NUM_FORMATS) - 1;
        if (r.formats == 0) r.formats = kAll;
        if (r.formats & ~kAll) fail(GS_ERR_INVALID_ARG, "candidate mask names an unknown format");
        if (r.mode < GS_SEL_MODEL || r.mode > GS_SEL_FIXED) fail(GS_ERR_INVALID_ARG, "bad selector mode");
        if (r.fixed < 0 || r.fixed >= GS_NUM_FORMATS) fail(GS_ERR_INVALID_ARG, "bad fixed format");
        if (r.max_bytes == 0) r.max_bytes = kDefaultMaxBytes;
        if (r.bsr_block == 0) r.bsr_block = kDefaultBsrBlock;
        if (r.bsr_block < 1 || r.bsr_block > 64) fail(GS_ERR_INVALID_ARG, "bsr_block outside 1..64");
        if (r.profile_reps <= 0) r.profile_reps = 3;
        gs_ctx_ *c = new gs_ctx_();
        try {
            c->opts = r;
            c->opts.model_path = nullptr;  // not retained
            if (r.mode == GS_SEL_MODEL) {  // the other modes never consult a model
                std::string text = kBuiltinModel;
                if (r.model_path) {
                    std::FILE *f = std::fopen(r.model_path, "rb");
                    if (!f) fail(GS_ERR_MODEL, "cannot open model file %s", r.model_path);
                    text.clear();
                    char buf[1 << 16];
                    size_t n;
                    while ((n = std::fread(buf, 1, sizeof buf, f)) > 0) text.append(buf, n);
                    const bool bad = std::ferror(f) != 0;
                    std::fclose(f);
                    if (bad) fail(GS_ERR_MODEL, "cannot read model file %s", r.model_path);
                }
                parse_model(text, c->model);
            }
        } catch (...) {
            delete c;
            throw;
        }
        *out = c;
    });
}

void gs_ctx_destroy(gs_ctx c) { delete c; }

int gs_select(gs_ctx c, uint64_t key, const gs_coo *A, int64_t F, gs_stream stream, int32_t *chosen)
{
    return guarded([&] {
        if (!c) fail(GS_ERR_INVALID_ARG, "null context");
        if (F <= 0) fail(GS_ERR_INVALID_ARG, "F must be positive");
        if (c->opts.mode == GS_SEL_PROFILE)
            fail(GS_ERR_INVALID_ARG, "profiling selection needs X and Y: use gs_select_and_run");
        hipStream_t s = (hipStream_t)stream;
        Entry &e = lookup(*c, key, A, s);
        int f = choose(*c, e, F, nullptr, 0, nullptr, 0, s);
        if (chosen) *chosen = f;
    });
}

int gs_select_and_run(gs_ctx c, uint64_t key, const gs_coo *A, const float *X, int64_t ldx,
                      float *Y, int64_t ldy, int64_t F, gs_stream stream, int32_t *chosen)
{
    return guarded([&] {
        if (!c) fail(GS_ERR_INVALID_ARG, "null context");
        hipStream_t s = (hipStream_t)stream;
        Entry &e = lookup(*c, key, A, s);
        check_spmm_args(e.built[GS_CSR], X, ldx, Y, ldy, F);
        const int f = choose(*c, e, F, X, ldx, Y, ldy, s);
        run_spmm(*e.built[f], X, ldx, Y, ldy, F, s);
        if (chosen) *chosen = f;
    });
}

int gs_ctx_stats(gs_ctx c, gs_select_stats *out)
{
    if (!c || !out) {
        set_error("gs_ctx_stats: null argument");
        return GS_ERR_INVALID_ARG;
    }
    *out = c->last;
    return GS_OK;
}

}  // extern "C"
