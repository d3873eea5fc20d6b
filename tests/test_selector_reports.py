"""The predictor reports reproduce from the committed profiles (CPU only):

* selector/comparison.md -- the comparison selectors of Table 3 (Sec. 6.2)
  and Fig. 11 (Sec. 6.4): decision tree, 1-nearest neighbour, SVM and MLP
  beside the shipped gradient-boosted trees, each cross-validated on the same
  profiled samples with fixed seeds.  Accuracy, speedup over CSR and fraction
  of the profiling oracle must match the table (prediction times are host
  timings and are not compared).
* selector/generalisation.md -- the shipped model on the held-out matrices
  with random float values.
"""
import os
import re

import pytest

from conftest import ROOT

SEL = os.path.join(ROOT, "paper_2111_00352_amd", "selector")

pytest.importorskip("sklearn")


def _table(path):
    rows = {}
    for line in open(path):
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 4 and re.match(r"^[0-9.]+$", cells[1]):
            rows[cells[0]] = cells[1:]
    return rows


def test_comparison_table_reproduces():
    from paper_2111_00352_amd.selector import compare

    table = _table(os.path.join(SEL, "comparison.md"))
    rows, n_samples, _ = compare.compare(os.path.join(SEL, "data.csv"), folds=5, timing=False)
    assert f"on {n_samples} profiled" in open(os.path.join(SEL, "comparison.md")).read()
    assert {r[0] for r in rows} == set(table)
    for name, acc, sp, frac, orac, bad, _ in rows:
        t_acc, t_sp, t_frac, t_bad = table[name][:4]
        assert abs(acc - float(t_acc)) <= 0.006, (name, acc, t_acc)
        assert abs(sp - float(t_sp.rstrip("x"))) <= 0.004, (name, sp, t_sp)
        assert abs(frac - float(t_frac)) <= 0.004, (name, frac, t_frac)
        assert bad == int(t_bad), name
    gbt = next(r for r in rows if r[0] == "gradient-boosted trees")
    # the shipped predictor leads on accuracy, as XGBoost does in the paper (Sec. 6.4)
    assert gbt[1] == max(r[1] for r in rows)


def test_generalisation_table_reproduces():
    import numpy as np

    from paper_2111_00352_amd.selector import train

    X, T, groups, _ = train.load(os.path.join(SEL, "data.csv"))
    mn, mx = X.min(axis=0), X.max(axis=0)
    clf = train.fit(train.normalise(X, mn, mx), train.labels(T))
    Xe, Te, _, _ = train.load(os.path.join(SEL, "eval.csv"))
    pe = clf.predict(train.normalise(Xe, mn, mx))
    acc = float((pe == train.labels(Te)).mean())
    sp, frac, orac, bad = train.evaluate(Te, pe)
    row = _table(os.path.join(SEL, "generalisation.md"))["all"]
    assert int(row[0]) == len(pe)
    assert abs(acc - float(row[1])) <= 0.006 and abs(sp - float(row[2].rstrip("x"))) <= 0.004
    assert abs(frac - float(row[4])) <= 0.004 and bad == int(row[5])
    # the exported model file predicts the same classes as the trained model
    mn2, mx2, base, classes, trees = train.read_model(os.path.join(SEL, "model.gsm"))
    S = train.score_exported(trees, base, train.normalise(Xe, mn2, mx2))
    assert (np.array([classes[i] for i in np.argmax(S, axis=1)]) ==
            np.array([train.FMT_IDS[train.TIE_ORDER[c]] for c in pe])).all()
