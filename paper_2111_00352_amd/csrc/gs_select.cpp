// Per-layer format selection and dispatch (Sec. 4, Sec. 4.6): features are
// extracted once per adjacency key (Sec. 4.4), min-max normalised and
// clipped with the model's training range, scored by a boosted tree
// ensemble (Sec. 4.1; one score per candidate format, highest wins), the
// matrix is converted only when the chosen format has not been built for
// this key yet, and the chosen format's kernel runs.

#include <algorithm>
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

#include "gs_host.h"
#include "gs_internal.h"

namespace gs {
gs_matrix_ *build_csr(const gs_coo *A, const gs_build_opts &o, hipStream_t s, bool plan);
void check_coo(const gs_coo *A);
}  // namespace gs

using namespace gs;

namespace {

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

// Eq. 1 over the profiled candidates: the smallest w R + (1 - w) M, with
// the running time R and the device bytes M min-max scaled over the
// candidates; within 1e-4 of the smallest counts as optimal and the first in
// tie order is taken.
int eq1_choice(const Entry &e, uint32_t cand, double w)
{
    double tmin = 1e300, tmax = -1e300, mmin = 1e300, mmax = -1e300;
    for (int fmt : kTieOrder)
        if (cand & (1u << fmt)) {
            tmin = std::min(tmin, e.prof_time[fmt]);
            tmax = std::max(tmax, e.prof_time[fmt]);
            mmin = std::min(mmin, (double)e.bytes[fmt]);
            mmax = std::max(mmax, (double)e.bytes[fmt]);
        }
    auto scaled = [](double v, double lo, double hi) { return hi > lo ? (v - lo) / (hi - lo) : 0.0; };
    double O[GS_NUM_FORMATS], best = 1e300;
    for (int fmt : kTieOrder)
        if (cand & (1u << fmt)) {
            O[fmt] = w * scaled(e.prof_time[fmt], tmin, tmax) + (1.0 - w) * scaled((double)e.bytes[fmt], mmin, mmax);
            best = std::min(best, O[fmt]);
        }
    for (int fmt : kTieOrder)
        if ((cand & (1u << fmt)) && O[fmt] <= best + 1e-4) return fmt;
    return GS_CSR;
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
            uint32_t cand = 0;
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
                    cand |= 1u << fmt;
                    if (t < best * 0.99) {  // within 1%: keep the earlier one in tie order
                        best = t;
                        chosen = fmt;
                    }
                }
                if (c.opts.mem_weight > 0.0 && cand) chosen = eq1_choice(e, cand, 1.0 - c.opts.mem_weight);
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
        gs_selector_opts r = {GS_SEL_MODEL, GS_CSR, nullptr, kDefaultMaxBytes, kDefaultBsrBlock, 3, 0, 0.0};
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
        if (!(r.mem_weight >= 0.0 && r.mem_weight <= 1.0))
            fail(GS_ERR_INVALID_ARG, "mem_weight outside [0, 1]");
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
                std::string err;
                if (!parse_model(text, c->model, &err)) fail(GS_ERR_MODEL, "%s", err.c_str());
                // the model's labels fix its trade-off of Eq. 1
                if (std::fabs((1.0 - r.mem_weight) - c->model.w) > 1e-9)
                    fail(GS_ERR_MODEL, "the model was trained for w = %g, the context asks for w = %g",
                         c->model.w, 1.0 - r.mem_weight);
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
