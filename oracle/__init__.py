"""CPU oracle for the GNN aggregation SpMM, its storage formats and features.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the GPU library (``paper_2111_00352_amd``) and the library never imports
it.

The arithmetic lives in ``oracle.c`` (plain loops, fp64 SpMM accumulation);
this module only compiles it with gcc and marshals numpy arrays.  Each wrapper
names the passage of the paper (arXiv 2111.00352) it follows:

* storage formats COO/CSR/CSC/DIA/BSR ........ Sec. 2.2 (ELL: padded row packing)
* SpMM Y = A.X ................................ Sec. 2.1
* features F1..F19 ............................ Sec. 4.4, Table 2
* two-layer GCN forward / backward (gcn.py) ... Sec. 2.1, Sec. 5.1 (numpy fp64)

``check_spmm`` applies the acceptance bound |Y - Y_ref| <= 1e-5 * (|A|.|X|) + 1e-6
elementwise, evaluated in fp64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, ERR_ARG, ERR_INDEX, ERR_DUPLICATE, ERR_EXPLICIT_ZERO = 0, -1, -2, -3, -4

FEATURE_NAMES = [
    "numRow", "numCol", "NNZ", "N_diags", "aver_RD", "max_RD", "min_RD", "dev_RD",
    "aver_CD", "max_CD", "min_CD", "dev_CD", "ER_DIA", "ER_CD", "row_bounce",
    "col_bounce", "density", "cv", "max_mu",
]
INT_NAMES = [
    "n_rows", "n_cols", "nnz", "n_diags", "max_rd", "min_rd", "max_cd", "min_cd",
    "sum_rd2", "sum_cd2", "bounce_r", "bounce_c", "n_blocks16",
]


# ORACLE_SANITIZE=1: a separate build with AddressSanitizer and
# UndefinedBehaviorSanitizer (the process must preload the ASan runtime).
_SANITIZE = os.environ.get("ORACLE_SANITIZE") == "1"
if _SANITIZE:
    _LIB = os.path.join(_HERE, "liboracle_san.so")
_SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so with gcc (OpenMP for the SpMM loop)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        opt = _SAN_FLAGS if _SANITIZE else ["-O2"]
        subprocess.check_call(
            ["gcc", *opt, "-fopenmp", "-std=c11", "-Wall", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        sig = {
            "or_canon": (ctypes.c_int, [i64, i64, i64, p, p, p, p, p, p]),
            "or_csr": (ctypes.c_int, [i64, i64, p, p]),
            "or_ell_width": (i64, [i64, p]),
            "or_ell": (ctypes.c_int, [i64, i64, p, p, p, p, p]),
            "or_ell_to_coo": (i64, [i64, i64, p, p, p, p, p]),
            "or_dia_offsets": (i64, [i64, i64, i64, p, p, p]),
            "or_dia": (ctypes.c_int, [i64, i64, p, i64, p, p, p, p]),
            "or_dia_to_coo": (i64, [i64, i64, i64, p, p, p, p, p]),
            "or_bsr_structure": (i64, [i64, i64, i64, i64, p, p, p, p]),
            "or_bsr_values": (ctypes.c_int, [i64, i64, p, p, i64, i64, p, p, p, p]),
            "or_bsr_to_coo": (i64, [i64, i64, i64, p, p, p, p, p, p]),
            "or_features": (ctypes.c_int, [i64, i64, i64, p, p, p, p]),
            "or_spmm": (ctypes.c_int, [i64, p, p, p, p, i64, i64, p, p]),
            "or_spmm_rows": (ctypes.c_int, [i64, p, p, p, p, p, i64, i64, p, p]),
            "or_spmm64": (ctypes.c_int, [i64, p, p, p, p, i64, i64, p]),
            "or_num_threads": (ctypes.c_int, []),
            "or_set_threads": (None, [ctypes.c_int]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__("oracle error %d" % code)
        self.code = code


def canon(R, C, row, col, val):
    """Canonical COO (Sec. 2.2 COO): validated and sorted by (row, col)."""
    row, col, val = _i32(row), _i32(col), _f32(val)
    Z = row.size
    orow = np.empty(Z, np.int32)
    ocol = np.empty(Z, np.int32)
    oval = np.empty(Z, np.float32)
    rc = lib().or_canon(R, C, Z, _p(row), _p(col), _p(val), _p(orow), _p(ocol), _p(oval))
    if rc != OK:
        raise OracleError(rc)
    return orow, ocol, oval


def csr(R, crow):
    """CSR row pointers (Sec. 2.2 CSR) from canonical COO rows."""
    crow = _i32(crow)
    rp = np.empty(R + 1, np.int32)
    lib().or_csr(R, crow.size, _p(crow), _p(rp))
    return rp


def csc(R, C, row, col, val):
    """CSC (Sec. 2.2): (col_ptr[C+1], row[Z], val[Z]) in (col, row) order --
    by definition the CSR arrays of the transpose."""
    ocol, orow, oval = canon(C, R, col, row, val)
    return csr(C, ocol), orow, oval


def ell(R, row_ptr, col, val):
    """ELL: (K, ell_col[K*R], ell_val[K*R]) column-major, padding (-1, +0.0f)."""
    row_ptr, col, val = _i32(row_ptr), _i32(col), _f32(val)
    K = lib().or_ell_width(R, _p(row_ptr))
    ec = np.empty(K * R, np.int32)
    ev = np.empty(K * R, np.float32)
    lib().or_ell(R, K, _p(row_ptr), _p(col), _p(val), _p(ec), _p(ev))
    return int(K), ec, ev


def ell_to_coo(R, K, ell_col, ell_val, nnz_hint):
    ell_col, ell_val = _i32(ell_col), _f32(ell_val)
    n = max(nnz_hint, 0)
    r = np.empty(n, np.int32); c = np.empty(n, np.int32); v = np.empty(n, np.float32)
    z = lib().or_ell_to_coo(R, K, _p(ell_col), _p(ell_val), _p(r), _p(c), _p(v))
    assert z == n, (z, n)
    return r, c, v


def dia(R, C, crow, ccol, cval):
    """DIA (Sec. 2.2 DIA): (offsets ascending, data[N_diags*R] row-indexed)."""
    crow, ccol, cval = _i32(crow), _i32(ccol), _f32(cval)
    Z = crow.size
    nd = lib().or_dia_offsets(R, C, Z, _p(crow), _p(ccol), None)
    off = np.empty(max(nd, 0), np.int32)
    lib().or_dia_offsets(R, C, Z, _p(crow), _p(ccol), _p(off))
    data = np.empty(nd * R, np.float32)
    lib().or_dia(R, nd, _p(off), Z, _p(crow), _p(ccol), _p(cval), _p(data))
    return off, data


def dia_to_coo(R, C, offsets, data, nnz_hint):
    offsets, data = _i32(offsets), _f32(data)
    n = nnz_hint
    r = np.empty(n, np.int32); c = np.empty(n, np.int32); v = np.empty(n, np.float32)
    z = lib().or_dia_to_coo(R, C, offsets.size, _p(offsets), _p(data), _p(r), _p(c), _p(v))
    assert z == n, (z, n)
    return r, c, v


def bsr(R, C, b, crow, ccol, cval):
    """BSR(b) (Sec. 2.2 BSR): (block_ptr, block_col, block_val[nb*b*b])."""
    crow, ccol, cval = _i32(crow), _i32(ccol), _f32(cval)
    Z = crow.size
    nbr = (R + b - 1) // b
    nb = lib().or_bsr_structure(R, C, b, Z, _p(crow), _p(ccol), None, None)
    bp = np.empty(nbr + 1, np.int32)
    bc = np.empty(nb, np.int32)
    lib().or_bsr_structure(R, C, b, Z, _p(crow), _p(ccol), _p(bp), _p(bc))
    bv = np.empty(nb * b * b, np.float32)
    lib().or_bsr_values(R, b, _p(bp), _p(bc), nb, Z, _p(crow), _p(ccol), _p(cval), _p(bv))
    return bp, bc, bv


def bsr_to_coo(R, C, b, block_ptr, block_col, block_val, nnz_hint):
    bp, bc, bv = _i32(block_ptr), _i32(block_col), _f32(block_val)
    n = nnz_hint
    r = np.empty(n, np.int32); c = np.empty(n, np.int32); v = np.empty(n, np.float32)
    z = lib().or_bsr_to_coo(R, C, b, _p(bp), _p(bc), _p(bv), _p(r), _p(c), _p(v))
    assert z == n, (z, n)
    return r, c, v


def features(R, C, crow, ccol):
    """Features F1..F19 (Sec. 4.4, Table 2) plus the integer aggregates."""
    crow, ccol = _i32(crow), _i32(ccol)
    ints = np.zeros(13, np.int64)
    f = np.zeros(19, np.float64)
    rc = lib().or_features(R, C, crow.size, _p(crow), _p(ccol), _p(ints), _p(f))
    if rc != OK:
        raise OracleError(rc)
    return dict(zip(INT_NAMES, (int(x) for x in ints))), f


def spmm(R, row_ptr, col, val, X):
    """SpMM (Sec. 2.1) in fp64: returns (Y64, M) with M = |A|.|X|."""
    row_ptr, col, val = _i32(row_ptr), _i32(col), _f32(val)
    X = _f32(X)
    F = X.shape[1] if X.ndim == 2 else 1
    Y = np.empty((R, F), np.float64)
    M = np.empty((R, F), np.float64)
    lib().or_spmm(R, _p(row_ptr), _p(col), _p(val), _p(X), F, F, _p(Y), _p(M))
    return Y, M


def spmm64(R, row_ptr, col, val, X):
    """SpMM (Sec. 2.1) of an fp64 dense operand, summed in fp64: Y64[R, F]."""
    row_ptr, col, val = _i32(row_ptr), _i32(col), _f32(val)
    X = np.ascontiguousarray(X, dtype=np.float64)
    F = X.shape[1]
    Y = np.empty((R, F), np.float64)
    lib().or_spmm64(R, _p(row_ptr), _p(col), _p(val), _p(X), F, F, _p(Y))
    return Y


def spmm_rows(rows, row_ptr, col, val, X):
    """SpMM (Sec. 2.1) for the listed rows only: (Y64[len(rows),F], M)."""
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    row_ptr, col, val = _i32(row_ptr), _i32(col), _f32(val)
    X = _f32(X)
    F = X.shape[1]
    Y = np.empty((rows.size, F), np.float64)
    M = np.empty((rows.size, F), np.float64)
    lib().or_spmm_rows(rows.size, _p(rows), _p(row_ptr), _p(col), _p(val), _p(X), F, F, _p(Y), _p(M))
    return Y, M


def num_threads() -> int:
    return int(lib().or_num_threads())


def set_threads(n: int) -> None:
    """Thread count of the parallel SpMM loop (results are identical for any n)."""
    lib().or_set_threads(int(n))


def spmm_bound(M):
    """Acceptance bound per element: 1e-5 * (|A|.|X|) + 1e-6."""
    return 1e-5 * M + 1e-6


def check_spmm(Y, Yref, M):
    """Return (ok, worst ratio |err|/bound); NaN anywhere is a failure."""
    Y = np.asarray(Y, dtype=np.float64)
    err = np.abs(Y - Yref)
    ratio = err / spmm_bound(M)
    worst = float(np.max(ratio)) if ratio.size else 0.0
    ok = bool(np.all(np.isfinite(Y) == np.isfinite(Yref))) and (ratio.size == 0 or worst <= 1.0)
    return ok, worst
