"""DOK / LIL host construction formats (Sec. 2.2): round trips, and the
triplets they produce are the canonical COO the oracle defines."""
import json
import os

import numpy as np

import graphgen
import oracle
from conftest import GOLDEN
from paper_2111_00352_amd import hostfmt


def _w1():
    with open(os.path.join(GOLDEN, "w1_5x5.json")) as f:
        return json.load(f)


def test_w1_through_dok_and_lil():
    g = _w1()
    ent = list(zip(g["entries_row"], g["entries_col"], g["entries_val"]))
    dok = {(i, j): a for i, j, a in reversed(ent)}
    r, c, v = hostfmt.dok_to_coo(dok)
    assert r.tolist() == g["entries_row"] and c.tolist() == g["entries_col"]
    assert v.tolist() == g["entries_val"]
    # LIL by hand: row 3 empty, columns listed out of order within a row
    lil_cols = [[2, 0], [1], [4, 0, 3], [], [4]]
    lil_vals = [[2, 1], [3], [6, 4, 5], [], [7]]
    r2, c2, v2 = hostfmt.lil_to_coo(lil_cols, lil_vals)
    assert r2.tolist() == g["entries_row"] and c2.tolist() == g["entries_col"]
    assert v2.tolist() == g["entries_val"]
    cols, vals = hostfmt.coo_to_lil(g["R"], r2, c2, v2)
    assert cols == [[0, 2], [1], [0, 3, 4], [], [4]] and vals == [[1, 2], [3], [4, 5, 6], [], [7]]


def test_random_round_trips_match_oracle_canonical_order():
    R, C = 300, 200
    row, col, val = graphgen.random_coo(R, C, 2000, 17, empty_rows=0.2)
    row, col, val = graphgen.shuffled(row, col, val, 18)
    cr, cc, cv = oracle.canon(R, C, row, col, val)
    r, c, v = hostfmt.dok_to_coo(hostfmt.coo_to_dok(row, col, val))
    assert np.array_equal(r, cr) and np.array_equal(c, cc) and np.array_equal(v, cv)
    cols, vals = hostfmt.coo_to_lil(R, row, col, val)
    r, c, v = hostfmt.lil_to_coo(cols, vals)
    assert np.array_equal(r, cr) and np.array_equal(c, cc) and np.array_equal(v, cv)


def test_empty_and_malformed():
    r, c, v = hostfmt.dok_to_coo({})
    assert r.size == c.size == v.size == 0
    try:
        hostfmt.lil_to_coo([[0, 1]], [[1.0]])
    except ValueError:
        pass
    else:
        raise AssertionError("ragged LIL row accepted")
