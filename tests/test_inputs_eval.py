"""The held-out evaluation matrices (random float values): sizes and
densities inside their stated ranges, canonical order, no stored zeros,
reproducible from the seed."""
import numpy as np

import graphgen


def test_evaluation_matrices_are_canonical_and_in_range():
    lo, hi = graphgen.EVAL_SIZE_RANGE
    for i in (0, 7, 31, 99):
        n, row, col, val, meta = graphgen.evaluation_matrix(i)
        assert lo <= n <= hi and meta["kind"] == "random-float"
        assert row.size >= 1 and row.size <= graphgen.TRAIN_NNZ_CAP
        keys = row.astype(np.int64) * n + col
        assert (np.diff(keys) > 0).all()  # sorted by (row, col), no duplicates
        assert (row >= 0).all() and (row < n).all() and (col >= 0).all() and (col < n).all()
        assert val.dtype == np.float32 and (val > 0).all() and (val <= 1).all()
        n2, row2, col2, val2, _ = graphgen.evaluation_matrix(i)
        assert n2 == n and (row2 == row).all() and (col2 == col).all() and (val2 == val).all()
