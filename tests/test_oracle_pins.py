"""Pins of the CPU oracle against facts fixed outside it.

Each test ties the oracle to something the paper or plain mathematics fixes:
a hand-worked example (tests/golden/w1_5x5.json), the density the paper prints
for an identity-like 34x34 matrix (Table 1, KarateClub row: 2.94%), dense
brute-force products, closed forms of GCN normalisation, of row-stochastic
matrices and of the 2-D grid, exact special cases (identity, diagonal), and
independent numpy constructions of every storage layout and integer count.
"""
import json
import math
import os

import numpy as np
import pytest

import graphgen
import oracle
from conftest import GOLDEN


def _w1():
    with open(os.path.join(GOLDEN, "w1_5x5.json")) as f:
        return json.load(f)


def _dense(R, C, row, col, val):
    A = np.zeros((R, C), np.float64)
    A[row, col] = val
    return A


# ---------------------------------------------------------------- W1 example

def test_w1_layouts():
    g = _w1()
    R, C = g["R"], g["C"]
    row, col, val = (np.array(g[k]) for k in ("entries_row", "entries_col", "entries_val"))
    r, c, v = oracle.canon(R, C, row[::-1], col[::-1], val[::-1])
    assert (r == row).all() and (c == col).all() and (v == val).all()
    rp = oracle.csr(R, r)
    assert rp.tolist() == g["csr_row_ptr"]
    K, ec, ev = oracle.ell(R, rp, c, v)
    assert K == g["ell_K"] and ec.tolist() == g["ell_col"] and ev.tolist() == g["ell_val"]
    off, data = oracle.dia(R, C, r, c, v)
    assert off.tolist() == g["dia_offsets"] and data.tolist() == g["dia_data"]
    bp, bc, bv = oracle.bsr(R, C, g["bsr_b"], r, c, v)
    assert bp.tolist() == g["bsr_block_ptr"]
    assert bc.tolist() == g["bsr_block_col"]
    assert bv.tolist() == g["bsr_block_val"]
    cp, cr, cv = oracle.csc(R, C, row[::-1], col[::-1], val[::-1])
    assert cp.tolist() == g["csc_col_ptr"] and cr.tolist() == g["csc_row"] and cv.tolist() == g["csc_val"]


def test_w1_padding_is_positive_zero():
    g = _w1()
    R, C = g["R"], g["C"]
    r, c, v = oracle.canon(R, C, g["entries_row"], g["entries_col"], g["entries_val"])
    _, ec, ev = oracle.ell(R, oracle.csr(R, r), c, v)
    assert (ev.view(np.uint32)[ec == -1] == 0).all()
    _, data = oracle.dia(R, C, r, c, v)
    assert (data.view(np.uint32)[data == 0] == 0).all()


def test_w1_features():
    g = _w1()
    R, C = g["R"], g["C"]
    ints, f = oracle.features(R, C, np.array(g["entries_row"]), np.array(g["entries_col"]))
    assert ints == g["ints"]
    assert f.tolist() == g["features"]  # bit-exact doubles


def test_w1_spmm_ones():
    g = _w1()
    R, C = g["R"], g["C"]
    r, c, v = np.array(g["entries_row"]), np.array(g["entries_col"]), np.array(g["entries_val"])
    rp = oracle.csr(R, r)
    Y, M = oracle.spmm(R, rp, c, v, np.ones((C, 1), np.float32))
    assert Y[:, 0].tolist() == g["spmm_ones_F1"]
    assert M[:, 0].tolist() == g["spmm_ones_F1"]  # all values positive, X = 1


# --------------------------------------------------- the paper's printed value

def test_identity_34_density_matches_karateclub_row():
    # Table 1 prints 2.94% for the 34 x 34 KarateClub input: 34 nonzeros of
    # 34*34, i.e. an identity-like matrix.
    n = 34
    idx = np.arange(n)
    ints, f = oracle.features(n, n, idx, idx)
    assert round(100 * f[16], 2) == 2.94
    assert f[16] == 1.0 / 34
    # identity special case of every other feature
    assert ints["n_diags"] == 1 and ints["max_rd"] == ints["min_rd"] == 1
    assert f[12] == 1.0 and f[13] == 1.0  # ER_DIA, ER_CD
    assert f[7] == 0.0 and f[11] == 0.0 and f[17] == 0.0  # devs, cv
    assert f[14] == 0.0 and f[15] == 0.0  # bounces
    assert f[18] == 0.0


# ------------------------------------------------------------ SpMM pins

@pytest.mark.parametrize("R,C,nnz,F,seed", [
    (1, 1, 1, 1, 0), (7, 5, 12, 3, 1), (64, 40, 300, 17, 2), (129, 257, 2000, 64, 3),
    (300, 300, 0, 5, 4), (50, 1, 30, 2, 5), (1, 60, 40, 9, 6),
])
def test_spmm_dense_bruteforce(R, C, nnz, F, seed):
    row, col, val = graphgen.random_coo(R, C, nnz, seed, empty_rows=0.2)
    X = graphgen.features_x(C, F, seed + 100, "normal")
    rp = oracle.csr(R, row)
    Y, M = oracle.spmm(R, rp, col, val, X)
    A = _dense(R, C, row, col, val.astype(np.float64))
    Yd = A @ X.astype(np.float64)
    Md = np.abs(A) @ np.abs(X.astype(np.float64))
    assert np.all(np.abs(Y - Yd) <= 1e-12 * Md + 1e-300)
    assert np.allclose(M, Md, rtol=1e-12, atol=0)


def test_spmm_nonsymmetric_orientation():
    # Y_i aggregates row i over columns j (Y = A X, not A^T X)
    row, col, val = np.array([0]), np.array([2]), np.array([5.0], np.float32)
    X = np.array([[1.0], [10.0], [100.0]], np.float32)
    Y, _ = oracle.spmm(3, oracle.csr(3, row), col, val, X)
    assert Y[:, 0].tolist() == [500.0, 0.0, 0.0]


def test_spmm_identity_and_diagonal_exact():
    n, F = 97, 13
    idx = np.arange(n, dtype=np.int32)
    X = graphgen.features_x(n, F, 7, "normal")
    Y, _ = oracle.spmm(n, oracle.csr(n, idx), idx, np.ones(n, np.float32), X)
    assert (Y == X.astype(np.float64)).all()
    d = graphgen.features_x(n, 1, 8, "normal")[:, 0]
    d[d == 0] = 1
    Y, _ = oracle.spmm(n, oracle.csr(n, idx), idx, d, X)
    assert (Y == d.astype(np.float64)[:, None] * X.astype(np.float64)).all()


def test_spmm_linearity():
    g = graphgen.scaled(3)
    rp = oracle.csr(g.R, g.row)
    X1 = graphgen.features_x(g.C, 8, 11)
    X2 = graphgen.features_x(g.C, 8, 12)
    Y1, M1 = oracle.spmm(g.R, rp, g.col, g.val, X1)
    Y2, M2 = oracle.spmm(g.R, rp, g.col, g.val, X2)
    Y3, _ = oracle.spmm(g.R, rp, g.col, g.val, (X1.astype(np.float64) + X2).astype(np.float32))
    X3 = (X1.astype(np.float64) + X2).astype(np.float32)
    # X1 + X2 is exact in fp32 here (both are multiples of 2^-23 in [-1,1))
    assert (X3.astype(np.float64) == X1.astype(np.float64) + X2).all()
    assert np.all(np.abs(Y3 - (Y1 + Y2)) <= 1e-13 * (M1 + M2))


def test_gcn_rowsum_closed_form():
    # GCN values a_ij = 1/sqrt(d_i d_j): with X = 1, Y_i = d_i^-1/2 * sum_j d_j^-1/2.
    g = graphgen.config(1)
    d = np.bincount(g.row, minlength=g.R).astype(np.float64)
    rp = oracle.csr(g.R, g.row)
    Y, _ = oracle.spmm(g.R, rp, g.col, g.val, np.ones((g.C, 1), np.float32))
    closed = np.zeros(g.R)
    np.add.at(closed, g.row, 1.0 / np.sqrt(d[g.col]))
    closed /= np.sqrt(d)
    # values are fp32 roundings of the exact weights: each term within 2^-24 relative
    assert np.all(np.abs(Y[:, 0] - closed) <= 2.0**-24 * closed * 1.0001)


def test_gcn_eigenvector_closed_form():
    # D^-1/2 (A+I) D^-1/2 maps D^1/2 1 to itself.
    g = graphgen.config(1)
    d = np.bincount(g.row, minlength=g.R).astype(np.float64)
    x = np.sqrt(d).astype(np.float32)[:, None]
    Y, _ = oracle.spmm(g.R, oracle.csr(g.R, g.row), g.col, g.val, x)
    assert np.all(np.abs(Y[:, 0] - np.sqrt(d)) <= 3 * 2.0**-24 * np.sqrt(d) + 1e-12)


def test_row_stochastic_rows_sum_to_one():
    g = graphgen.scaled(5)
    rp = oracle.csr(g.R, g.row)
    Y, _ = oracle.spmm(g.R, rp, g.col, g.val, np.ones((g.C, 1), np.float32))
    r = np.diff(rp).astype(np.float64)
    assert np.all(np.abs(Y[:, 0] - 1.0) <= r * 2.0**-24 + 1e-15)


def test_spmm_rows_matches_full():
    g = graphgen.scaled(2)
    rp = oracle.csr(g.R, g.row)
    Y, M = oracle.spmm(g.R, rp, g.col, g.val, g.X)
    rows = np.array([0, 5, g.R - 1, int(np.argmax(np.diff(rp)))])
    Ys, Ms = oracle.spmm_rows(rows, rp, g.col, g.val, g.X)
    assert (Ys == Y[rows]).all() and (Ms == M[rows]).all()


def test_check_spmm_bound():
    Yref = np.array([[1.0, -2.0]])
    M = np.array([[1.0, 2.0]])
    ok, w = oracle.check_spmm(np.array([[1.0 + 1.0e-5, -2.0]]), Yref, M)
    assert ok and w <= 1.0
    ok, _ = oracle.check_spmm(np.array([[1.0 + 2.0e-5, -2.0]]), Yref, M)
    assert not ok
    ok, _ = oracle.check_spmm(np.array([[np.nan, -2.0]]), Yref, M)
    assert not ok


# ------------------------------------------------ canonical COO and errors

def test_canon_sorts_shuffled_input():
    g = graphgen.scaled(2)
    r, c, v = graphgen.shuffled(g.row, g.col, g.val, 5)
    orow, ocol, oval = oracle.canon(g.R, g.C, r, c, v)
    assert (orow == g.row).all() and (ocol == g.col).all()
    assert (oval.view(np.uint32) == g.val.view(np.uint32)).all()


def test_canon_errors_and_precedence():
    R = C = 4
    ok_r, ok_c, ok_v = [0, 1, 2], [0, 1, 2], [1.0, 2.0, 3.0]
    with pytest.raises(oracle.OracleError) as e:
        oracle.canon(R, C, [0, 4], [0, 0], [1.0, 1.0])
    assert e.value.code == oracle.ERR_INDEX
    with pytest.raises(oracle.OracleError) as e:
        oracle.canon(R, C, [0, -1], [0, 0], [1.0, 1.0])
    assert e.value.code == oracle.ERR_INDEX
    with pytest.raises(oracle.OracleError) as e:
        oracle.canon(R, C, [0, 1], [0, 0], [1.0, -0.0])
    assert e.value.code == oracle.ERR_EXPLICIT_ZERO
    with pytest.raises(oracle.OracleError) as e:
        oracle.canon(R, C, [1, 0, 1], [2, 0, 2], [1.0, 1.0, 2.0])
    assert e.value.code == oracle.ERR_DUPLICATE
    # index beats zero beats duplicate
    with pytest.raises(oracle.OracleError) as e:
        oracle.canon(R, C, [1, 1, 9], [2, 2, 0], [0.0, 1.0, 1.0])
    assert e.value.code == oracle.ERR_INDEX
    with pytest.raises(oracle.OracleError) as e:
        oracle.canon(R, C, [1, 1], [2, 2], [0.0, 1.0])
    assert e.value.code == oracle.ERR_EXPLICIT_ZERO
    oracle.canon(R, C, ok_r, ok_c, ok_v)
    oracle.canon(R, C, [], [], [])


# ----------------------------------- layouts vs independent numpy builders

def _np_ell(R, row, col, val):
    cnt = np.bincount(row, minlength=R)
    K = int(cnt.max()) if row.size else 0
    start = np.concatenate([[0], np.cumsum(cnt)])
    k = np.arange(row.size) - start[row]
    ec = np.full(K * R, -1, np.int32)
    ev = np.zeros(K * R, np.float32)
    ec[k * R + row] = col
    ev[k * R + row] = val
    return K, ec, ev


def _np_dia(R, row, col, val):
    diff = col.astype(np.int64) - row
    off = np.unique(diff)
    data = np.zeros(off.size * R, np.float32)
    data[np.searchsorted(off, diff) * R + row] = val
    return off.astype(np.int32), data


def _np_bsr(R, C, b, row, col, val):
    nbr = -(-R // b)
    keys = np.unique((row // b).astype(np.int64) * (C // b + 2) + col // b)
    kbr = keys // (C // b + 2)
    kbc = keys % (C // b + 2)
    bp = np.searchsorted(kbr, np.arange(nbr + 1)).astype(np.int32)
    blk = np.searchsorted(keys, (row // b).astype(np.int64) * (C // b + 2) + col // b)
    bv = np.zeros(keys.size * b * b, np.float32)
    bv[blk * b * b + (row % b) * b + col % b] = val
    return bp, kbc.astype(np.int32), bv


CASES = [
    (1, 1, 1, 0), (5, 7, 9, 1), (33, 17, 100, 2), (100, 100, 0, 3), (257, 129, 3000, 4),
    (16, 16, 256, 5), (31, 64, 400, 6), (1000, 999, 8000, 7),
]


@pytest.mark.parametrize("R,C,nnz,seed", CASES)
def test_layouts_match_numpy_and_round_trip(R, C, nnz, seed):
    row, col, val = graphgen.random_coo(R, C, nnz, seed, empty_rows=0.15)
    Z = row.size
    rp = oracle.csr(R, row)
    assert (np.diff(rp) == np.bincount(row, minlength=R)).all()
    K, ec, ev = oracle.ell(R, rp, col, val)
    K2, ec2, ev2 = _np_ell(R, row, col, val)
    assert K == K2 and (ec == ec2).all() and (ev.view(np.uint32) == ev2.view(np.uint32)).all()
    r, c, v = oracle.ell_to_coo(R, K, ec, ev, Z)
    assert (r == row).all() and (c == col).all() and (v == val).all()
    off, data = oracle.dia(R, C, row, col, val)
    off2, data2 = _np_dia(R, row, col, val)
    assert (off == off2).all() and (data.view(np.uint32) == data2.view(np.uint32)).all()
    r, c, v = oracle.dia_to_coo(R, C, off, data, Z)
    assert (r == row).all() and (c == col).all() and (v == val).all()
    for b in (1, 2, 3, 16):
        bp, bc, bv = oracle.bsr(R, C, b, row, col, val)
        bp2, bc2, bv2 = _np_bsr(R, C, b, row, col, val)
        assert (bp == bp2).all() and (bc == bc2).all()
        assert (bv.view(np.uint32) == bv2.view(np.uint32)).all()
        r, c, v = oracle.bsr_to_coo(R, C, b, bp, bc, bv, Z)
        assert (r == row).all() and (c == col).all() and (v == val).all()


# ---------------------------------------------- features vs independent counts

@pytest.mark.parametrize("R,C,nnz,seed", CASES)
def test_feature_integers_match_numpy(R, C, nnz, seed):
    row, col, _ = graphgen.random_coo(R, C, nnz, seed, empty_rows=0.15)
    ints, f = oracle.features(R, C, row, col)
    rc = np.bincount(row, minlength=R).astype(np.int64)
    cc = np.bincount(col, minlength=C).astype(np.int64)
    exp = dict(
        n_rows=R, n_cols=C, nnz=row.size,
        n_diags=int(np.unique(col.astype(np.int64) - row).size),
        max_rd=int(rc.max()), min_rd=int(rc.min()), max_cd=int(cc.max()), min_cd=int(cc.min()),
        sum_rd2=int((rc * rc).sum()), sum_cd2=int((cc * cc).sum()),
        bounce_r=int(np.abs(np.diff(rc)).sum()), bounce_c=int(np.abs(np.diff(cc)).sum()),
        n_blocks16=int(np.unique((row // 16).astype(np.int64) * (C // 16 + 1) + col // 16).size),
    )
    assert ints == exp
    # structural invariants of the doubles
    assert f[0] == R and f[1] == C and f[2] == row.size
    if row.size:
        assert math.isclose(f[4] * R, row.size, rel_tol=1e-15)
        assert math.isclose(f[8] * C, row.size, rel_tol=1e-15)
        assert f[7] >= 0 and f[11] >= 0
        assert math.isclose(f[7], float(np.std(rc)), rel_tol=1e-12, abs_tol=1e-15)
        assert math.isclose(f[11], float(np.std(cc)), rel_tol=1e-12, abs_tol=1e-15)
        assert 0 < f[12] <= 1 and 0 < f[13] <= 1


def test_symmetric_pattern_row_equals_column_features():
    g = graphgen.scaled(4)
    ints, f = oracle.features(g.R, g.C, g.row, g.col)
    assert ints["max_rd"] == ints["max_cd"] and ints["sum_rd2"] == ints["sum_cd2"]
    assert f[4:8].tolist() == f[8:12].tolist()
    assert f[14] == f[15]


def test_empty_matrix_features():
    ints, f = oracle.features(10, 12, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert ints["nnz"] == 0 and ints["n_diags"] == 0 and ints["n_blocks16"] == 0
    assert f.tolist() == [10.0, 12.0] + [0.0] * 17


def _grid(m):
    n = m * m
    ids = np.arange(n)
    r, c = ids // m, ids % m
    rows, cols = [ids], [ids]
    for dr, dc in ((-1, 0), (1, 0), (0, -1), (0, 1)):
        ok = (r + dr >= 0) & (r + dr < m) & (c + dc >= 0) & (c + dc < m)
        rows.append(ids[ok])
        cols.append(ids[ok] + dr * m + dc)
    row = np.concatenate(rows)
    col = np.concatenate(cols)
    o = np.lexsort((col, row))
    return n, row[o].astype(np.int32), col[o].astype(np.int32)


@pytest.mark.parametrize("m", [16, 48, 512])
def test_grid_closed_forms(m):
    n, row, col = _grid(m)
    ints, f = oracle.features(n, n, row, col)
    nbr = m * m // 16
    exp = dict(
        n_rows=n, n_cols=n, nnz=5 * m * m - 4 * m, n_diags=5, max_rd=5, min_rd=3, max_cd=5,
        min_cd=3, sum_rd2=4 * 9 + 4 * (m - 2) * 16 + (m - 2) ** 2 * 25,
        sum_cd2=4 * 9 + 4 * (m - 2) * 16 + (m - 2) ** 2 * 25,
        bounce_r=2 * m + 2, bounce_c=2 * m + 2,
        n_blocks16=nbr + 2 * (nbr - m) + 2 * (nbr - m // 16),
    )
    assert ints == exp
    off, _ = oracle.dia(n, n, row, col, np.ones(row.size, np.float32))
    assert off.tolist() == [-m, -1, 0, 1, m]
    if m == 512:
        with open(os.path.join(GOLDEN, "mesh_512.json")) as fh:
            gold = json.load(fh)
        assert ints == gold["ints"]
        names = oracle.FEATURE_NAMES
        for k, v in gold["features"].items():
            assert f[names.index(k)] == v, k


def test_mesh_generator_matches_grid():
    g = graphgen.config(3)
    n, row, col = _grid(512)
    assert (g.row == row).all() and (g.col == col).all()
    assert (g.val > 0).all() and (g.val <= 1).all()


@pytest.mark.parametrize("R,C,nnz,seed", [(40, 25, 200, 3), (7, 90, 60, 4), (64, 64, 0, 5)])
def test_csc_is_the_column_compressed_dense_matrix(R, C, nnz, seed):
    # brute force: walking the dense matrix column by column, top to bottom
    row, col, val = graphgen.random_coo(R, C, nnz, seed, empty_rows=0.2)
    cp, cr, cv = oracle.csc(R, C, *graphgen.shuffled(row, col, val, seed + 1))
    A = _dense(R, C, row, col, val)
    exp_ptr, exp_row, exp_val = [0], [], []
    for j in range(C):
        nz = np.nonzero(A[:, j])[0]
        exp_row += nz.tolist()
        exp_val += A[nz, j].tolist()
        exp_ptr.append(exp_ptr[-1] + nz.size)
    assert cp.tolist() == exp_ptr and cr.tolist() == exp_row
    assert np.array_equal(cv.astype(np.float64), np.array(exp_val, dtype=np.float64))
