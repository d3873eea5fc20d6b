"""Compare format predictors on the profiled training data.

Usage: python -m paper_2111_00352_amd.selector.compare [DATA.csv] [--folds 5] [--md OUT.md]

The paper sets its gradient-boosted trees against a decision tree and a CNN
from prior format-selection work (Sec. 5.2, Sec. 6.2 and its table of
inference time, accuracy and realised speedup) and against an MLP, 1-nearest
neighbour and an SVM (Sec. 6.4, accuracy and prediction time).  Every
candidate here sees the same inputs (Table 2 features plus the 16x16 block
fill and F, min-max scaled with the training fold's range and clipped) and
the same labels (Eq. 1 with w = 1, 3% ties) as ``train``, and is scored with
the same grouped k-fold split (no matrix in both the training and the test
fold) on:
  * accuracy against the profiled label;
  * geometric-mean speedup of the chosen format over fixed CSR, and the
    fraction of the profiling oracle's performance (Sec. 6.3);
  * the time of one prediction (one feature vector, the selector's use),
    median over repeated single-sample calls of the scikit-learn model.
The CNN (which reads the matrix as an image) is not included: its input is
not the feature vector the library extracts.
"""
import argparse
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from paper_2111_00352_amd.selector import DATA_PATH  # noqa: E402
from paper_2111_00352_amd.selector import train  # noqa: E402


def candidates(seed=0):
    from sklearn.neighbors import KNeighborsClassifier
    from sklearn.neural_network import MLPClassifier
    from sklearn.svm import SVC
    from sklearn.tree import DecisionTreeClassifier

    return {
        "gradient-boosted trees": lambda: _Fitted(train.fit, seed),
        "decision tree": lambda: DecisionTreeClassifier(random_state=seed),
        "1-nearest neighbour": lambda: KNeighborsClassifier(n_neighbors=1),
        "SVM (RBF)": lambda: SVC(C=10.0, gamma="scale", random_state=seed),
        "MLP (64-64)": lambda: MLPClassifier(hidden_layer_sizes=(64, 64), max_iter=2000,
                                             random_state=seed),
    }


class _Fitted:
    """Adapter so the shipped trainer fits like a scikit-learn estimator."""

    def __init__(self, fn, seed):
        self.fn, self.seed, self.clf = fn, seed, None

    def fit(self, X, y):
        self.clf = self.fn(X, y, self.seed)
        return self

    def predict(self, X):
        return self.clf.predict(X)


def predict_time(model, Xn, reps=200):
    ts = []
    for i in range(reps):
        x = Xn[i % len(Xn)][None, :]
        t0 = time.perf_counter()
        model.predict(x)
        ts.append(time.perf_counter() - t0)
    return float(np.median(ts))


def compare(data=DATA_PATH, folds=5, timing=True):
    """Cross-validates every candidate predictor: rows of (name, accuracy,
    speedup over CSR, fraction of oracle, oracle over CSR, infeasible picks,
    median one-prediction time in s or None)."""
    from sklearn.model_selection import GroupKFold

    X, T, groups, kinds = train.load(data)
    y = train.labels(T)
    rows = []
    for name, make in candidates().items():
        pred = np.zeros_like(y)
        tpred = []
        for tr, te in GroupKFold(n_splits=folds).split(X, y, groups):
            mn, mx = X[tr].min(axis=0), X[tr].max(axis=0)
            m = make().fit(train.normalise(X[tr], mn, mx), y[tr])
            Xte = train.normalise(X[te], mn, mx)
            pred[te] = m.predict(Xte)
            if timing:
                tpred.append(predict_time(m, Xte, reps=50))
        acc = float((pred == y).mean())
        sp, frac, orac, bad = train.evaluate(T, pred)
        rows.append((name, acc, sp, frac, orac, bad, float(np.median(tpred)) if timing else None))
    return rows, len(y), len(set(groups))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("data", nargs="?", default=DATA_PATH)
    ap.add_argument("--folds", type=int, default=5)
    ap.add_argument("--md", help="also write the table as markdown to this file")
    a = ap.parse_args()
    rows, n_samples, n_matrices = compare(a.data, a.folds)
    for name, acc, sp, frac, orac, bad, tp in rows:
        print(f"{name:24s} accuracy {acc:.3f}  speedup over CSR {sp:.3f}x (oracle {orac:.3f}x)  "
              f"fraction of oracle {frac:.3f}  infeasible picks {bad}  predict {tp * 1e6:.0f} us", flush=True)
    if a.md:
        lines = [f"Predictor comparison on {n_samples} profiled (matrix, F) samples from "
                 f"{n_matrices} matrices, {a.folds}-fold grouped cross-validation "
                 "(`python -m paper_2111_00352_amd.selector.compare`).", "",
                 "| predictor | accuracy | speedup over CSR (geo-mean) | fraction of oracle | "
                 "infeasible picks | one prediction (scikit-learn, host) |",
                 "|---|---|---|---|---|---|"]
        for name, acc, sp, frac, orac, bad, tp in rows:
            lines.append(f"| {name} | {acc:.3f} | {sp:.3f}x | {frac:.3f} | {bad} | {tp * 1e6:.0f} us |")
        lines.append("")
        lines.append(f"Profiling oracle (always the fastest format): {rows[0][4]:.3f}x over CSR.")
        with open(a.md, "w") as fh:
            fh.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
