"""GNN-aggregation SpMM with per-layer sparse-format selection on MI355X.

A thin ctypes binding over ``libgnnspmm.so`` (HIP kernels for gfx950 behind
the C ABI of ``include/gnnspmm.h``).  This module only marshals arguments:
validation, conversion, feature extraction, selection and every SpMM run in
the library.  PyTorch supplies device memory (its caching allocator is
installed as the library's allocator) and streams (the current stream).

Paper: Qiu, You, Wang, "Optimizing Sparse Matrix Multiplications for Graph
Neural Networks", arXiv 2111.00352 -- storage formats Sec. 2.2, SpMM Sec. 2.1,
features Sec. 4.4 / Table 2, the per-layer ``SpMMPredict`` runtime Sec. 4.6.

There is no fallback: if the library is missing or no GPU is present, calls
raise.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "FORMATS", "FORMAT_NAMES", "GnnSpmmError", "Matrix", "SelectContext", "build_format",
    "extract_features", "lib", "library_path", "FEATURE_NAMES", "set_allocator",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libgnnspmm.so")

FORMATS = {"coo": 0, "csr": 1, "ell": 2, "dia": 3, "bsr": 4, "csc": 5}
FORMAT_NAMES = {v: k for k, v in FORMATS.items()}
FEATURE_NAMES = [
    "numRow", "numCol", "NNZ", "N_diags", "aver_RD", "max_RD", "min_RD", "dev_RD",
    "aver_CD", "max_CD", "min_CD", "dev_CD", "ER_DIA", "ER_CD", "row_bounce",
    "col_bounce", "density", "cv", "max_mu",
]
SEL_MODES = {"model": 0, "profile": 1, "fixed": 2}

_i64, _u64, _i32, _p = ctypes.c_int64, ctypes.c_uint64, ctypes.c_int32, ctypes.c_void_p


class _Coo(ctypes.Structure):
    _fields_ = [("n_rows", _i64), ("n_cols", _i64), ("nnz", _i64),
                ("row", _p), ("col", _p), ("val", _p)]


class _BuildOpts(ctypes.Structure):
    _fields_ = [("bsr_block", _i32), ("assume_canonical", _i32), ("max_bytes", _u64)]


class _Info(ctypes.Structure):
    _fields_ = [("format", _i32), ("bsr_block", _i32), ("n_rows", _i64), ("n_cols", _i64),
                ("nnz", _i64), ("param", _i64), ("device_bytes", _u64)]


class _Features(ctypes.Structure):
    _fields_ = [("n_rows", _i64), ("n_cols", _i64), ("nnz", _i64), ("n_diags", _i64),
                ("max_rd", _i64), ("min_rd", _i64), ("max_cd", _i64), ("min_cd", _i64),
                ("sum_rd2", _u64), ("sum_cd2", _u64), ("bounce_r", _u64), ("bounce_c", _u64),
                ("n_blocks16", _i64), ("f", ctypes.c_double * 19)]


class _SelOpts(ctypes.Structure):
    _fields_ = [("mode", _i32), ("fixed", _i32), ("model_path", ctypes.c_char_p),
                ("max_bytes", _u64), ("bsr_block", _i32), ("profile_reps", _i32),
                ("formats", ctypes.c_uint32), ("mem_weight", ctypes.c_double)]


class _SelStats(ctypes.Structure):
    _fields_ = [("t_features", ctypes.c_double), ("t_predict", ctypes.c_double),
                ("t_convert", ctypes.c_double), ("chosen", _i32), ("feasible_mask", _i32),
                ("scores", ctypes.c_double * len(FORMATS))]


_ALLOC_FN = ctypes.CFUNCTYPE(_p, ctypes.c_size_t, _p, _p)
_FREE_FN = ctypes.CFUNCTYPE(None, _p, _p, _p)


class _Allocator(ctypes.Structure):
    _fields_ = [("alloc", _ALLOC_FN), ("free", _FREE_FN), ("ctx", _p)]


class GnnSpmmError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"gnnspmm error {code}: {msg}")
        self.code = code


ERR_INVALID_ARG, ERR_INDEX, ERR_DUPLICATE, ERR_EXPLICIT_ZERO = -1, -2, -3, -4
ERR_INFEASIBLE, ERR_OOM, ERR_HIP, ERR_MODEL, ERR_UNSUPPORTED = -5, -6, -7, -8, -9

_lib = None
_alloc_keep = None
# Every hook set ever installed through set_allocator, kept for the life of
# the process: the library frees each buffer through the hooks that
# allocated it, so a collected callback would be called after it is gone.
_hooks_alive: list = []


def library_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """Loads libgnnspmm.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(
            f"{_LIB_PATH} is missing: build it with `python -m paper_2111_00352_amd.build`"
        )
    L = ctypes.CDLL(_LIB_PATH)
    c_int = ctypes.c_int
    P = ctypes.POINTER
    sigs = {
        "gs_set_allocator": (c_int, [P(_Allocator)]),
        "gs_build_format": (c_int, [P(_Coo), c_int, P(_BuildOpts), _p, P(_p), P(_u64)]),
        "gs_convert": (c_int, [_p, c_int, P(_BuildOpts), _p, P(_p), P(_u64)]),
        "gs_spmm": (c_int, [_p, _p, _i64, _p, _i64, _i64, _p]),
        "gs_spmm_noalloc": (c_int, [_p, _p, _i64, _p, _i64, _i64, _p]),
        "gs_to_coo": (c_int, [_p, _p, _p, _p, _p]),
        "gs_get_info": (c_int, [_p, P(_Info)]),
        "gs_get_array": (c_int, [_p, c_int, P(_p), P(_u64)]),
        "gs_copy_array": (c_int, [_p, c_int, _p, _u64, _p]),
        "gs_destroy": (None, [_p]),
        "gs_extract_features": (c_int, [P(_Coo), P(_BuildOpts), _p, P(_Features)]),
        "gs_matrix_features": (c_int, [_p, _p, P(_Features)]),
        "gs_ctx_create": (c_int, [P(_SelOpts), P(_p)]),
        "gs_ctx_destroy": (None, [_p]),
        "gs_select": (c_int, [_p, _u64, P(_Coo), _i64, _p, P(_i32)]),
        "gs_select_and_run": (c_int, [_p, _u64, P(_Coo), _p, _i64, _p, _i64, _i64, _p, P(_i32)]),
        "gs_ctx_stats": (c_int, [_p, P(_SelStats)]),
        "gs_last_error": (ctypes.c_char_p, []),
        "gs_abi_version": (c_int, []),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(rc: int):
    if rc != 0:
        raise GnnSpmmError(rc, lib().gs_last_error().decode(errors="replace"))


def _require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("gnnspmm needs a ROCm GPU (torch.cuda.is_available() is False)")
    _install_torch_allocator()


def _install_torch_allocator(reinstall: bool = False):
    """Routes the library's device allocations through PyTorch's caching allocator."""
    global _alloc_keep
    if _alloc_keep is not None:
        if reinstall:
            _check(lib().gs_set_allocator(ctypes.byref(_alloc_keep[0])))
        return

    def _alloc(nbytes, stream, _ctx):
        try:
            return torch.cuda.caching_allocator_alloc(int(nbytes), stream=int(stream or 0))
        except Exception:  # out of memory -> the library reports GS_ERR_OOM
            return None

    def _free(ptr, _stream, _ctx):
        torch.cuda.caching_allocator_delete(int(ptr))

    a = _Allocator(_ALLOC_FN(_alloc), _FREE_FN(_free), None)
    _check(lib().gs_set_allocator(ctypes.byref(a)))
    _alloc_keep = (a, _alloc, _free)


def set_allocator(alloc=None, free=None):
    """Installs device allocation hooks for all later library allocations
    (gs_set_allocator).  alloc(nbytes, stream) returns a device pointer
    (int) aligned to 256 bytes, or 0 / None when it cannot allocate;
    free(ptr, stream) releases one; both must be stream-ordered (see
    gs_allocator).  No arguments reinstall PyTorch's caching allocator.

    Buffers always go back through the hooks that allocated them, so the
    hooks must outlive every handle built with them: this binding keeps each
    hook set (the callables and their ctypes wrappers) referenced until the
    process ends, whatever the caller does with its own references."""
    if (alloc is None) != (free is None):
        raise ValueError("alloc and free must both be given or both be None")
    if alloc is None:
        _install_torch_allocator(reinstall=True)
        return

    def _a(nbytes, stream, _ctx):
        try:
            p = alloc(int(nbytes), int(stream or 0))
        except Exception:  # reported by the library as GS_ERR_OOM
            return None
        return int(p) if p else None

    def _f(ptr, stream, _ctx):
        free(int(ptr), int(stream or 0))

    hooks = _Allocator(_ALLOC_FN(_a), _FREE_FN(_f), None)
    _hooks_alive.append((hooks, _a, _f, alloc, free))
    _check(lib().gs_set_allocator(ctypes.byref(hooks)))


def _stream(stream=None) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream if hasattr(stream, "cuda_stream") else stream)


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None or t.numel() == 0 else t.data_ptr()


def _coo_struct(row, col, val, shape):
    for t, dt in ((row, torch.int32), (col, torch.int32), (val, torch.float32)):
        if not t.is_cuda or t.dtype != dt or not t.is_contiguous() or t.dim() != 1:
            raise ValueError("row/col must be contiguous CUDA int32, val contiguous CUDA float32")
    if not (row.numel() == col.numel() == val.numel()):
        raise ValueError("row, col and val must have the same length")
    R, C = int(shape[0]), int(shape[1])
    return _Coo(R, C, row.numel(), _ptr(row), _ptr(col), _ptr(val))


def _opts(bsr_block=16, assume_canonical=False, max_bytes=None):
    return _BuildOpts(int(bsr_block), 1 if assume_canonical else 0, int(max_bytes or 0))


def _check_dense(X: torch.Tensor, name: str):
    if not X.is_cuda or X.dtype != torch.float32 or X.dim() != 2 or X.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D CUDA float32 tensor with unit column stride")


class Matrix:
    """A sparse matrix held on the device in one storage format."""

    def __init__(self, handle: int):
        self._h = ctypes.c_void_p(handle)
        info = _Info()
        _check(lib().gs_get_info(self._h, ctypes.byref(info)))
        self.format = FORMAT_NAMES[info.format]
        self.shape = (info.n_rows, info.n_cols)
        self.nnz = info.nnz
        self.param = info.param
        self.bsr_block = info.bsr_block
        self.device_bytes = info.device_bytes

    @property
    def handle(self) -> ctypes.c_void_p:
        return self._h

    def close(self):
        if self._h:
            lib().gs_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def spmm(self, X: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
        """Y = A.X (Sec. 2.1), asynchronous on the current stream."""
        _check_dense(X, "X")
        R, C = self.shape
        if X.shape[0] != C:
            raise ValueError(f"X has {X.shape[0]} rows, A has {C} columns")
        F = X.shape[1]
        if out is None:
            out = torch.empty((R, F), dtype=torch.float32, device=X.device)
        _check_dense(out, "out")
        if out.shape[0] != R or out.shape[1] != F:
            raise ValueError("out has the wrong shape")
        _check(lib().gs_spmm(self._h, _ptr(X), X.stride(0), _ptr(out), out.stride(0), F,
                             _stream(stream)))
        return out

    def spmm_noalloc(self, X: torch.Tensor, out: torch.Tensor, stream=None) -> torch.Tensor:
        """Y = A.X into the preallocated `out` without any device allocation
        (gs_spmm_noalloc: the workspace is the library's fixed per-device
        scratch array, shared by every such call on the device)."""
        _check_dense(X, "X")
        _check_dense(out, "out")
        R, C = self.shape
        if X.shape[0] != C or out.shape[0] != R or out.shape[1] != X.shape[1]:
            raise ValueError("X / out shapes do not match A")
        _check(lib().gs_spmm_noalloc(self._h, _ptr(X), X.stride(0), _ptr(out), out.stride(0), X.shape[1],
                                     _stream(stream)))
        return out

    def to_coo(self, stream=None):
        dev = torch.device("cuda", torch.cuda.current_device())
        row = torch.empty(self.nnz, dtype=torch.int32, device=dev)
        col = torch.empty(self.nnz, dtype=torch.int32, device=dev)
        val = torch.empty(self.nnz, dtype=torch.float32, device=dev)
        _check(lib().gs_to_coo(self._h, _ptr(row), _ptr(col), _ptr(val), _stream(stream)))
        return row, col, val

    def array(self, which: int, dtype=None, stream=None) -> torch.Tensor:
        """Copy of raw array `which` (see gs_get_array) as a 1-D tensor."""
        p, nbytes = ctypes.c_void_p(), _u64()
        _check(lib().gs_get_array(self._h, which, ctypes.byref(p), ctypes.byref(nbytes)))
        if dtype is None:
            dtype = torch.float32 if self._is_value_array(which) else torch.int32
        item = torch.empty((), dtype=dtype).element_size()
        out = torch.empty(nbytes.value // item, dtype=dtype,
                          device=torch.device("cuda", torch.cuda.current_device()))
        _check(lib().gs_copy_array(self._h, which, _ptr(out), nbytes.value, _stream(stream)))
        return out

    def _is_value_array(self, which: int) -> bool:
        f = self.format
        return (which == 2) or (which == 1 and f in ("ell", "dia"))

    def features(self, stream=None) -> dict:
        out = _Features()
        _check(lib().gs_matrix_features(self._h, _stream(stream), ctypes.byref(out)))
        return _features_dict(out)

    def convert(self, fmt: str, bsr_block=16, max_bytes=None, stream=None) -> "Matrix":
        h, need = ctypes.c_void_p(), _u64()
        o = _opts(bsr_block, False, max_bytes)
        rc = lib().gs_convert(self._h, FORMATS[fmt], ctypes.byref(o), _stream(stream),
                              ctypes.byref(h), ctypes.byref(need))
        if rc != 0:
            e = GnnSpmmError(rc, lib().gs_last_error().decode(errors="replace"))
            e.bytes_required = need.value
            raise e
        return Matrix(h.value)


def build_format(row, col, val, shape, fmt: str = "csr", bsr_block: int = 16,
                 max_bytes: int | None = None, assume_canonical: bool = False,
                 stream=None) -> Matrix:
    """Builds A (COO on the device, any order) in format fmt (Sec. 2.2)."""
    _require_gpu()
    A = _coo_struct(row, col, val, shape)
    o = _opts(bsr_block, assume_canonical, max_bytes)
    h, need = ctypes.c_void_p(), _u64()
    rc = lib().gs_build_format(ctypes.byref(A), FORMATS[fmt], ctypes.byref(o), _stream(stream),
                               ctypes.byref(h), ctypes.byref(need))
    if rc != 0:
        e = GnnSpmmError(rc, lib().gs_last_error().decode(errors="replace"))
        e.bytes_required = need.value
        raise e
    return Matrix(h.value)


def _features_dict(out: _Features) -> dict:
    d = {k: int(getattr(out, k)) for k, _ in _Features._fields_ if k != "f"}
    d["f"] = [float(x) for x in out.f]
    return d


def extract_features(row, col, val, shape, stream=None) -> dict:
    """Features F1..F19 of Table 2 (Sec. 4.4) plus the integer aggregates."""
    _require_gpu()
    A = _coo_struct(row, col, val, shape)
    out = _Features()
    _check(lib().gs_extract_features(ctypes.byref(A), None, _stream(stream), ctypes.byref(out)))
    return _features_dict(out)


class SelectContext:
    """Per-layer format selection and dispatch (the paper's SpMMPredict, Sec. 4.6)."""

    def __init__(self, mode: str = "model", fixed: str = "csr", model_path: str | None = None,
                 max_bytes: int | None = None, bsr_block: int = 16, profile_reps: int = 3,
                 formats=None, mem_weight: float = 0.0):
        """model_path None: the trained ensemble shipped in selector/model.gsm
        (the library's hand-set trees if that file is absent); "builtin": the
        hand-set trees.  formats: names of the candidate formats of "model"
        and "profile" (None: all).  mem_weight: 1 - w of Eq. 1, the weight of
        the memory footprint against the running time (0: time only); "model"
        needs a model trained for that w."""
        _require_gpu()
        if model_path is None:
            from paper_2111_00352_amd.selector import MODEL_PATH

            model_path = MODEL_PATH if os.path.exists(MODEL_PATH) else None
        elif model_path == "builtin":
            model_path = None
        self._model_path = model_path.encode() if model_path else None
        mask = 0 if formats is None else sum(1 << FORMATS[f] for f in formats)
        o = _SelOpts(SEL_MODES[mode], FORMATS[fixed], self._model_path, int(max_bytes or 0),
                     int(bsr_block), int(profile_reps), mask, float(mem_weight))
        h = ctypes.c_void_p()
        _check(lib().gs_ctx_create(ctypes.byref(o), ctypes.byref(h)))
        self._h = h
        self._keep = {}

    def close(self):
        if self._h:
            lib().gs_ctx_destroy(self._h)
            self._h = ctypes.c_void_p(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def run(self, key: int, row, col, val, shape, X: torch.Tensor,
            out: torch.Tensor | None = None, stream=None):
        """Y = A.X in the selected format; returns (Y, format name)."""
        _check_dense(X, "X")
        A = _coo_struct(row, col, val, shape)
        R = int(shape[0])
        F = X.shape[1]
        if out is None:
            out = torch.empty((R, F), dtype=torch.float32, device=X.device)
        _check_dense(out, "out")
        chosen = _i32()
        _check(lib().gs_select_and_run(self._h, int(key), ctypes.byref(A), _ptr(X), X.stride(0),
                                       _ptr(out), out.stride(0), F, _stream(stream),
                                       ctypes.byref(chosen)))
        return out, FORMAT_NAMES[chosen.value]

    def select(self, key: int, row, col, val, shape, F: int, stream=None) -> str:
        A = _coo_struct(row, col, val, shape)
        chosen = _i32()
        _check(lib().gs_select(self._h, int(key), ctypes.byref(A), int(F), _stream(stream),
                               ctypes.byref(chosen)))
        return FORMAT_NAMES[chosen.value]

    def stats(self) -> dict:
        st = _SelStats()
        _check(lib().gs_ctx_stats(self._h, ctypes.byref(st)))
        return dict(t_features=st.t_features, t_predict=st.t_predict, t_convert=st.t_convert,
                    chosen=FORMAT_NAMES.get(st.chosen, "?"), feasible_mask=st.feasible_mask,
                    scores={FORMAT_NAMES[i]: st.scores[i] for i in range(len(FORMATS))})
