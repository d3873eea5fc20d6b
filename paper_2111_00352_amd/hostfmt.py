"""Host-side construction formats of Sec. 2.2: DOK and LIL.

DOK (dictionary of keys) maps (row, col) to a value; LIL (list of lists)
keeps, per row, the column indices and values of that row's entries.  The
paper lists both among the candidate formats; neither is a layout a GPU
kernel traverses, so here they are what they are for in practice: ways to
assemble or edit a matrix incrementally on the host.  These helpers turn
them into the COO triplets the library takes (``build_format``,
``SelectContext.run``) and read a matrix back into them.  The triplets come
out in canonical (row, col) order; the library still validates them (index
range, explicit zeros, duplicates), so nothing here is trusted.
"""
from __future__ import annotations

import numpy as np


def _triplets(rows, cols, vals):
    row = np.asarray(rows, dtype=np.int32)
    col = np.asarray(cols, dtype=np.int32)
    val = np.asarray(vals, dtype=np.float32)
    order = np.lexsort((col, row))
    return row[order], col[order], val[order]


def dok_to_coo(dok: dict):
    """{(i, j): a} -> (row, col, val) sorted by (row, col)."""
    if not dok:
        return np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32)
    keys = list(dok.keys())
    return _triplets([k[0] for k in keys], [k[1] for k in keys], [dok[k] for k in keys])


def coo_to_dok(row, col, val) -> dict:
    """(row, col, val) -> {(i, j): a} (later duplicates overwrite earlier ones)."""
    return {(int(i), int(j)): float(a) for i, j, a in zip(np.asarray(row), np.asarray(col), np.asarray(val))}


def lil_to_coo(cols_per_row, vals_per_row):
    """Per-row column lists and value lists -> (row, col, val) sorted by (row, col)."""
    if len(cols_per_row) != len(vals_per_row):
        raise ValueError("LIL: one column list and one value list per row")
    rows, cols, vals = [], [], []
    for i, (cs, vs) in enumerate(zip(cols_per_row, vals_per_row)):
        if len(cs) != len(vs):
            raise ValueError(f"LIL row {i}: {len(cs)} columns but {len(vs)} values")
        rows += [i] * len(cs)
        cols += list(cs)
        vals += list(vs)
    return _triplets(rows, cols, vals)


def coo_to_lil(n_rows: int, row, col, val):
    """(row, col, val) -> (cols_per_row, vals_per_row), columns ascending."""
    row, col, val = _triplets(row, col, val)
    cuts = np.searchsorted(row, np.arange(n_rows + 1))
    cols = [col[cuts[i]:cuts[i + 1]].tolist() for i in range(n_rows)]
    vals = [val[cuts[i]:cuts[i + 1]].tolist() for i in range(n_rows)]
    return cols, vals
