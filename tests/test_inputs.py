"""The seeded input generators that only the big-offset parity tests use,
checked on the CPU: layouts as their docstrings state them."""
import numpy as np

import graphgen


def test_band_far_coo_layout():
    n = 101
    band = (-2, 0, 3)
    row, col, val = graphgen.band_far_coo(n, band, seed=5)
    keys = row.astype(np.int64) * n + col
    assert (np.diff(keys) > 0).all()  # canonical: sorted by (row, col), no duplicates
    exp = set()
    for i in range(n):
        exp.update((i, i + o) for o in band if 0 <= i + o < n)
        exp.add((i, (i + n // 2) % n))
    assert set(zip(row.tolist(), col.tolist())) == exp
    # the far diagonal switches offset at row n - n//2
    off = {(int(r), int(c)) for r, c in zip(row, col)}
    assert (n - n // 2 - 1, n - 1) in off and (n - n // 2, 0) in off
    # values: uniform [-1, 1) on the 2^-23 grid, never zero
    assert (val != 0).all() and (val >= -1).all() and (val < 1).all()
    assert np.array_equal(val * 2.0**23, np.round(val * 2.0**23))
    # seeded: the same seed gives the same values
    assert np.array_equal(graphgen.band_far_coo(n, band, seed=5)[2], val)


def test_structured_matrix_ranges():
    # the first 120 keep 10^4..2x10^5 rows, the next 40 reach 1.5x10^6
    small = [graphgen.structured_matrix(i)[0] for i in (0, 1, 2, 3)]
    assert all(1e4 <= n <= 2e5 for n in small)
    n, row, col, val, meta = graphgen.structured_matrix(123)
    assert 2e5 <= n <= 1.5e6 and meta["kind"] == "grid"
    assert (np.diff(row.astype(np.int64) * n + col) > 0).all() and (val == 1).all()
