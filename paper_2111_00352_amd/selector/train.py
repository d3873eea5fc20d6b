"""Train the format predictor from profiled data and export it.

Usage: python -m paper_2111_00352_amd.selector.train [DATA.csv] [--out model.gsm] [--w W]
           [--eval-csv eval.csv --eval-md generalisation.md] | [--importance importance.md] |
           [--w-sweep 0,0.25,... --md w_sweep.md]

Labels follow Eq. 1 with w = 1: the fastest format of each (matrix, F) row,
formats within 3% counting as tied and resolved in the order CSR < COO < ELL
< DIA < BSR.  The 3% is the run-to-run noise of the profiles (two
collections of the same kernels differ by 2-4% at the 90th percentile), so
a closer pair is not reliably ordered by one collection.  Features
(F1..F19 of Table 2, the 16x16 block fill, F) are min-max scaled to [0,1]
with the training range and clipped (Sec. 4.4), then rounded to fp32.  The
classifier is scikit-learn's gradient-boosted trees (xgboost is not
available); the ensemble is exported as per-class score trees and checked to
predict exactly as scikit-learn does.  Evaluation is grouped k-fold cross-
validation: a matrix is never in both the training and the test fold.
"""
import argparse
import csv
import math
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from paper_2111_00352_amd.selector import DATA_PATH, MODEL_PATH  # noqa: E402

FMT_IDS = {"coo": 0, "csr": 1, "ell": 2, "dia": 3, "bsr": 4}
TIE_ORDER = ["csr", "coo", "ell", "dia", "bsr"]
FEATS = ["numRow", "numCol", "NNZ", "N_diags", "aver_RD", "max_RD", "min_RD", "dev_RD",
         "aver_CD", "max_CD", "min_CD", "dev_CD", "ER_DIA", "ER_CD", "row_bounce",
         "col_bounce", "density", "cv", "max_mu"]


def load(path):
    with open(path) as fh:
        rows = list(csv.DictReader(fh))
    X, T, groups, kinds = [], [], [], []
    for r in rows:
        nb = float(r["n_blocks16"])
        x = [float(r[f]) for f in FEATS]
        x.append(float(r["NNZ"]) / (256.0 * nb) if nb > 0 else 0.0)
        x.append(float(r["F"]))
        X.append(x)
        T.append([float(r[f"t_{f}"]) for f in TIE_ORDER])
        groups.append(f"{r['set']}:{r['index']}")
        kinds.append(r["kind"])
    return np.array(X), np.array(T), np.array(groups), np.array(kinds)


TIE = 1.03  # times within 3% of the fastest count as tied


def labels(T):
    out = []
    for t in T:
        best = min(t)
        out.append(next(i for i, v in enumerate(t) if v <= best * TIE))
    return np.array(out)  # index into TIE_ORDER


def footprints(path):
    """Device bytes of every candidate format per sample (TIE_ORDER), from the
    profiled matrix's integer features -- the memory term M of Eq. 1.  Same
    sizes the library allocates: CSR 4(R+1)+8Z, COO 12Z, ELL 8 R max_RD,
    DIA 4 N_diags (R+1), BSR16 4(ceil(R/16)+1) + 1036 n_blocks16."""
    with open(path) as fh:
        rows = list(csv.DictReader(fh))
    M = []
    for r in rows:
        R, Z = float(r["numRow"]), float(r["NNZ"])
        nb, nd, k = float(r["n_blocks16"]), float(r["N_diags"]), float(r["max_RD"])
        M.append([4 * (R + 1) + 8 * Z, 12 * Z, 8 * R * k, 4 * nd * (R + 1),
                  4 * (math.ceil(R / 16) + 1) + (4 + 8 + 1024) * nb])
    return np.array(M)


def labels_eq1(T, M, w, tie=1e-4):
    """Eq. 1: the format minimising w R + (1 - w) M, with running time R and
    memory footprint M scaled to [0, 1] by the min and max over the whole
    profiled training set; formats within `tie` of the minimum count as
    optimal (Fig. 6 caption) and the earliest in TIE_ORDER is taken."""
    ok = np.isfinite(T)
    tmin, tmax = T[ok].min(), T[ok].max()
    mmin, mmax = M[ok].min(), M[ok].max()
    Tf, Mf = np.where(ok, T, tmin), np.where(ok, M, mmin)
    O = w * (Tf - tmin) / (tmax - tmin) + (1.0 - w) * (Mf - mmin) / (mmax - mmin)
    O = np.where(ok, O, np.inf)
    best = O.min(axis=1, keepdims=True)
    return np.argmax(O <= best + tie, axis=1)


def normalise(X, mn, mx):
    span = mx - mn
    Z = np.where(span > 0, (X - mn) / np.where(span > 0, span, 1), 0.0)
    return np.clip(Z, 0, 1).astype(np.float32).astype(np.float64)


def fit(Xn, y, seed=0):
    from sklearn.ensemble import GradientBoostingClassifier

    clf = GradientBoostingClassifier(n_estimators=80, max_depth=3, learning_rate=0.2,
                                     subsample=1.0, random_state=seed)
    clf.fit(Xn, y)
    return clf


def export(clf, mn, mx, path, w=1.0):
    classes = list(clf.classes_)
    K = len(classes)
    lr = clf.learning_rate
    base = clf._raw_predict_init(np.zeros((1, mn.size)))[0]
    trees = []
    est = clf.estimators_
    for stage in est:
        for k, tree in enumerate(stage):
            cls = k if K > 2 else 1
            t = tree.tree_
            nodes = []
            for i in range(t.node_count):
                if t.children_left[i] == -1:
                    nodes.append((-1, 0.0, 0, 0, lr * float(t.value[i][0][0])))
                else:
                    thr = float(np.nextafter(t.threshold[i], np.inf))  # x <= thr  ->  x < next(thr)
                    nodes.append((int(t.feature[i]), thr, int(t.children_left[i]),
                                  int(t.children_right[i]), 0.0))
            trees.append((cls, nodes))
    if K > 2:
        base_scores = list(base)
    else:
        base_scores = [0.0, float(base[0])]
    # version 2 of the model file: reals as exact hexadecimal literals,
    # leaves as "L value", internal nodes as "feat thr left right"
    hx = lambda v: float(v).hex()  # noqa: E731
    lines = ["GSMODEL 2", f"nfeat {mn.size}",
             "classes %d %s" % (K, " ".join(str(FMT_IDS[TIE_ORDER[c]]) for c in classes)),
             "min " + " ".join(hx(v) for v in mn),
             "max " + " ".join(hx(v) for v in mx),
             "base " + " ".join(hx(v) for v in base_scores),
             f"ntrees {len(trees)}"]
    for cls, nodes in trees:
        lines.append(f"tree {cls} {len(nodes)}")
        for f, thr, l, r, v in nodes:
            lines.append(f"L {hx(v)}" if f < 0 else f"{f} {hx(thr)} {l} {r}")
    if w != 1.0:  # the trade-off of Eq. 1 the labels were made for (1 when absent)
        lines.append(f"w {hx(w)}")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    return trees, base_scores, classes


def score_exported(trees, base_scores, Xn):
    S = np.tile(np.array(base_scores, dtype=np.float64), (Xn.shape[0], 1))
    for cls, nodes in trees:
        for r in range(Xn.shape[0]):
            i = 0
            while nodes[i][0] >= 0:
                f, thr, l, rr, _ = nodes[i]
                i = l if Xn[r, f] < thr else rr
            S[r, cls] += nodes[i][4]
    return S


def read_model(path):
    """The exported model file (version 1, decimal, or version 2, hexadecimal
    reals): (min, max, base scores, class format ids, trees), trees as
    written by ``export``."""
    with open(path) as fh:
        lines = [ln.split() for ln in fh if ln.strip()]
    head = {ln[0]: ln[1:] for ln in lines[:7]}
    assert lines[0] in (["GSMODEL", "1"], ["GSMODEL", "2"]), "not a model file"
    real = float if lines[0][1] == "1" else float.fromhex

    def node(tok):
        if tok[0] == "L":
            return (-1, 0.0, 0, 0, real(tok[1]))
        if len(tok) == 4:
            return (int(tok[0]), real(tok[1]), int(tok[2]), int(tok[3]), 0.0)
        f, t, l, r, v = tok
        return (int(f), real(t), int(l), int(r), real(v))

    mn = np.array([real(v) for v in head["min"]])
    mx = np.array([real(v) for v in head["max"]])
    base = [real(v) for v in head["base"]]
    classes = [int(v) for v in head["classes"][1:]]
    trees, i = [], 7
    for _ in range(int(head["ntrees"][0])):
        _, cls, n = lines[i]
        trees.append((int(cls), [node(t) for t in lines[i + 1:i + 1 + int(n)]]))
        i += 1 + int(n)
    return mn, mx, base, classes, trees


def model_input(f, n_blocks16, F):
    """The predictor's input for one (matrix, F): F1..F19 (Table 2 order),
    the 16x16 block fill, F -- as ``load`` builds it from the profiles."""
    nnz = float(f[FEATS.index("NNZ")])
    return list(map(float, f)) + [nnz / (256.0 * n_blocks16) if n_blocks16 > 0 else 0.0, float(F)]


def evaluate(T, pred):
    """Geometric-mean speedup over fixed CSR and fraction of the oracle."""
    tc = T[:, 0]
    tbest = T.min(axis=1)
    tsel = T[np.arange(len(pred)), pred]
    ok = np.isfinite(tsel)
    sp = np.exp(np.mean(np.log(tc[ok] / tsel[ok])))
    frac = np.exp(np.mean(np.log(tbest[ok] / tsel[ok])))
    orac = np.exp(np.mean(np.log(tc / tbest)))
    return sp, frac, orac, int((~ok).sum())


def cross_validate(X, y, groups, folds):
    from sklearn.model_selection import GroupKFold

    pred = np.zeros_like(y)
    for tr, te in GroupKFold(n_splits=folds).split(X, y, groups):
        mn, mx = X[tr].min(axis=0), X[tr].max(axis=0)
        pred[te] = fit(normalise(X[tr], mn, mx), y[tr]).predict(normalise(X[te], mn, mx))
    return pred


def w_sweep(a, X, T, groups, ws):
    """Sec. 6.5, impact of the optimisation goal: per w, the label mix and
    the cross-validated accuracy of a model trained for that w."""
    M = footprints(a.data)
    lines = [f"Eq. 1 labels per w on {len(X)} profiled samples ({len(set(groups))} matrices), "
             f"{a.folds}-fold grouped cross-validation "
             f"(`python -m paper_2111_00352_amd.selector.train --w-sweep ...`).", "",
             "| w | " + " | ".join(TIE_ORDER) + " | accuracy |", "|---" * (len(TIE_ORDER) + 2) + "|"]
    for w in ws:
        y = labels_eq1(T, M, w)
        counts = [int((y == c).sum()) for c in range(len(TIE_ORDER))]
        acc = float((cross_validate(X, y, groups, a.folds) == y).mean()) if len(set(y)) > 1 else 1.0
        print(f"w={w:.2f} labels " + ", ".join(f"{f}={n}" for f, n in zip(TIE_ORDER, counts))
              + f"  accuracy {acc:.3f}", flush=True)
        lines.append(f"| {w:.2f} | " + " | ".join(str(n) for n in counts) + f" | {acc:.3f} |")
    if a.md:
        with open(a.md, "w") as fh:
            fh.write("\n".join(lines) + "\n")


INPUT_NAMES = FEATS + ["bsr16_fill", "F"]


def importance(a, X, T, groups):
    """Fig. 7 analogue (Sec. 4.4): the cross-validated accuracy and fraction
    of the profiling oracle lost when one predictor input is left out, for
    each of the 21 inputs."""
    y = labels(T)
    base = cross_validate(X, y, groups, a.folds)
    acc0 = float((base == y).mean())
    frac0 = evaluate(T, base)[1]
    rows = []
    for i, name in enumerate(INPUT_NAMES):
        keep = [j for j in range(X.shape[1]) if j != i]
        pred = cross_validate(X[:, keep], y, groups, a.folds)
        acc = float((pred == y).mean())
        frac = evaluate(T, pred)[1]
        rows.append((name, acc0 - acc, frac0 - frac))
        print(f"without {name:12s} accuracy {acc:.3f} ({acc0 - acc:+.3f})  fraction of oracle {frac:.3f}",
              flush=True)
    rows.sort(key=lambda r: -r[1])
    lines = [f"Leave-one-out importance of the predictor's inputs on {len(y)} profiled samples "
             f"({len(set(groups))} matrices), {a.folds}-fold grouped cross-validation "
             "(`python -m paper_2111_00352_amd.selector.train --importance ...`): the drop in accuracy "
             f"and in fraction of the profiling oracle when the input is left out.  With every input: "
             f"accuracy {acc0:.3f}, fraction of oracle {frac0:.3f}.", "",
             "| input left out | accuracy drop | fraction-of-oracle drop |", "|---|---|---|"]
    for name, da, df in rows:
        lines.append(f"| {name} | {da:+.3f} | {df:+.4f} |")
    with open(a.importance, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def generalisation(a, clf, mn, mx):
    """The final model on held-out matrices with random float values
    (Sec. 5.1: generalisation to unseen sizes and sparsity): accuracy against
    the profiled label, speedup over fixed CSR and fraction of the profiling
    oracle (Sec. 6.3), overall and by size."""
    Xe, Te, ge, _ = load(a.eval_csv)
    ye = labels(Te)
    pe = clf.predict(normalise(Xe, mn, mx))
    acc = float((pe == ye).mean())
    sp, frac, orac, bad = evaluate(Te, pe)
    print(f"held-out set: {len(ye)} samples, {len(set(ge))} matrices; accuracy {acc:.3f}; speedup over CSR "
          f"{sp:.3f}x (oracle {orac:.3f}x); fraction of oracle {frac:.3f}; infeasible picks {bad}")
    n = Xe[:, FEATS.index("numRow")]
    lines = [f"The shipped model (trained on the profiled training set only) on {len(set(ge))} held-out matrices "
             f"with random float values, {len(ye)} (matrix, F) samples, profiled on the same kernels "
             "(`python -m paper_2111_00352_amd.selector.train --eval-csv selector/eval.csv ...`).", "",
             "| matrices | samples | accuracy | speedup over CSR (geo-mean) | profiling oracle over CSR | "
             "fraction of oracle | infeasible picks |", "|---|---|---|---|---|---|---|"]
    lines.append(f"| all | {len(ye)} | {acc:.3f} | {sp:.3f}x | {orac:.3f}x | {frac:.3f} | {bad} |")
    for lo, hi in ((0, 15001), (15001, 61000)):
        msk = (n >= lo) & (n < hi)
        if msk.sum():
            s2, f2, o2, b2 = evaluate(Te[msk], pe[msk])
            lab = "n <= 15,000 (training sizes)" if lo == 0 else "n > 15,000 (beyond them)"
            lines.append(f"| {lab} | {int(msk.sum())} | {float((pe[msk] == ye[msk]).mean()):.3f} | {s2:.3f}x | "
                         f"{o2:.3f}x | {f2:.3f} | {b2} |")
    counts = ", ".join(f"{TIE_ORDER[c]} {int((ye == c).sum())}" for c in range(len(TIE_ORDER)))
    lines += ["", f"Profiled labels: {counts}."]
    if a.eval_md:
        with open(a.eval_md, "w") as fh:
            fh.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("data", nargs="?", default=DATA_PATH)
    ap.add_argument("--out", default=MODEL_PATH)
    ap.add_argument("--folds", type=int, default=5)
    ap.add_argument("--w-sweep", help="comma-separated w values of Eq. 1: cross-validate a model per w "
                                      "(labels from time and memory) instead of exporting one")
    ap.add_argument("--md", help="with --w-sweep: also write the table as markdown")
    ap.add_argument("--importance", help="write the leave-one-out input importance table (markdown) "
                                         "instead of exporting a model")
    ap.add_argument("--eval-csv", help="held-out profiles: evaluate the exported model on them")
    ap.add_argument("--eval-md", help="with --eval-csv: write the evaluation table (markdown)")
    ap.add_argument("--w", type=float, default=1.0,
                    help="weight of Eq. 1 for the exported model's labels (1: time only, with 3%% ties); "
                         "a context uses it with mem_weight = 1 - w")
    a = ap.parse_args()
    from sklearn.model_selection import GroupKFold

    X, T, groups, kinds = load(a.data)
    if a.w_sweep:
        return w_sweep(a, X, T, groups, [float(v) for v in a.w_sweep.split(",")])
    if a.importance:
        return importance(a, X, T, groups)
    y = labels(T) if a.w == 1.0 else labels_eq1(T, footprints(a.data), a.w)
    print(f"{len(y)} samples, {len(set(groups))} matrices; label counts: "
          + ", ".join(f"{TIE_ORDER[c]}={int((y == c).sum())}" for c in range(5)))
    # cross-validation on unseen matrices
    pred = np.zeros_like(y)
    for tr, te in GroupKFold(n_splits=a.folds).split(X, y, groups):
        mn, mx = X[tr].min(axis=0), X[tr].max(axis=0)
        clf = fit(normalise(X[tr], mn, mx), y[tr])
        pred[te] = clf.predict(normalise(X[te], mn, mx))
    acc = float((pred == y).mean())
    sp, frac, orac, bad = evaluate(T, pred)
    print(f"cross-validated accuracy {acc:.3f}; speedup over CSR {sp:.3f}x (oracle {orac:.3f}x); "
          f"fraction of oracle performance {frac:.3f}; infeasible picks {bad}")
    for kd in sorted(set(kinds)):
        m = kinds == kd
        s2, f2, o2, _ = evaluate(T[m], pred[m])
        print(f"  {kd:10s} n={int(m.sum()):4d} acc {float((pred[m] == y[m]).mean()):.3f} "
              f"speedup {s2:.3f}x oracle {o2:.3f}x fraction {f2:.3f}")
    # final model on everything
    mn, mx = X.min(axis=0), X.max(axis=0)
    Xn = normalise(X, mn, mx)
    clf = fit(Xn, y)
    trees, base, classes = export(clf, mn, mx, a.out, w=a.w)
    S = score_exported(trees, base, Xn)
    ours = np.array([classes[i] for i in np.argmax(S, axis=1)])
    agree = float((ours == clf.predict(Xn)).mean())
    print(f"exported {len(trees)} trees to {a.out}; agreement with scikit-learn {agree:.4f}")
    if agree < 1.0:
        sys.exit("exported model disagrees with scikit-learn")
    if a.eval_csv:
        generalisation(a, clf, mn, mx)


if __name__ == "__main__":
    main()
