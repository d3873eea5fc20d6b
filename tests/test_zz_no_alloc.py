"""The allocation-free SpMM entry point (gs_spmm_noalloc) against gs_spmm.

gs_spmm_noalloc runs the same kernels as gs_spmm with the workspace taken from
the library's fixed per-device scratch array.  Checked through the C ABI:
  * its Y equals gs_spmm's bit for bit (CSC: within one fp32 step, its fp64
    atomics add in varying order) and lies within the SpMM bound of the
    oracle;
  * two calls in a row, the second with a smaller matrix and a narrower
    (ragged) F, so the second reuses scratch the first left behind;
  * no allocation happens during the call (PyTorch's allocator is the
    library's allocator, and its allocation count does not move);
  * COO handles and workspaces above the scratch size are refused with
    GS_ERR_UNSUPPORTED before any kernel runs.
"""
import ctypes

import numpy as np
import pytest
import torch

import graphgen
import oracle
import paper_2111_00352_amd as gs

pytestmark = pytest.mark.gpu

DEV = "cuda"
SCRATCH = 64 << 20  # GS_NOALLOC_SCRATCH_BYTES


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _bits(a):
    return np.ascontiguousarray(a).view(np.uint32)


def _hub_matrix(R, hubs, hub_len, base_nnz, seed):
    """Random canonical COO with `hubs` rows of hub_len entries (the CSR
    path's split rows, whose partial sums live in the workspace)."""
    rng = np.random.default_rng(seed)
    r0, c0, _ = graphgen.random_coo(R, R, base_nnz, seed)
    keys = [r0.astype(np.int64) * R + c0]
    for h in rng.choice(R, size=hubs, replace=False):
        keys.append(int(h) * R + rng.choice(R, size=hub_len, replace=False).astype(np.int64))
    keys = np.unique(np.concatenate(keys))
    row = (keys // R).astype(np.int32)
    col = (keys % R).astype(np.int32)
    val = rng.standard_normal(row.size).astype(np.float32)
    val[val == 0] = 0.5
    return row, col, val


def _noalloc(m, X, Y):
    L = gs.lib()
    return L.gs_spmm_noalloc(m.handle, X.data_ptr(), X.stride(0), Y.data_ptr(), Y.stride(0), X.shape[1],
                             torch.cuda.current_stream().cuda_stream)


def _allocations():
    return torch.cuda.memory_stats().get("allocation.all.allocated", 0)


def _check_pair(row, col, val, R, fmt, X, ldy_pad=0):
    F = X.shape[1]
    m = gs.build_format(_dev(row), _dev(col), _dev(val), (R, R), fmt)
    Xd = torch.zeros((R, F + 3), dtype=torch.float32, device=DEV)
    Xd[:, :F] = _dev(X)
    Xv = Xd[:, :F]
    Y_ref = m.spmm(Xv)  # the existing entry point (grows the handle's own workspace)
    Y = torch.full((R, F + ldy_pad), 7.0, dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    n0 = _allocations()
    rc = _noalloc(m, Xv, Y[:, :F])
    n1 = _allocations()
    assert rc == 0, gs.lib().gs_last_error()
    assert n1 == n0, "gs_spmm_noalloc allocated device memory"
    torch.cuda.synchronize()
    Yh, Rh = Y[:, :F].cpu().numpy(), Y_ref.cpu().numpy()
    if fmt == "csc":
        assert np.all(np.abs(Yh - Rh) <= np.spacing(np.abs(Rh).astype(np.float32)))
    else:
        assert (_bits(Yh) == _bits(Rh)).all(), f"{fmt}: differs from gs_spmm"
    if ldy_pad:
        assert (Y[:, F:].cpu().numpy() == 7.0).all()
    rp = oracle.csr(R, row)
    Yo, M = oracle.spmm(R, rp, col, val, X)
    ok, worst = oracle.check_spmm(Yh, Yo, M)
    assert ok, f"{fmt}: worst |err|/bound {worst}"
    m.close()


@pytest.mark.parametrize("fmt", ["csr", "csc", "ell", "dia", "bsr"])
def test_noalloc_matches_spmm_twice_second_smaller(fmt):
    # first call: hub rows of 3,000 entries (split across workgroups, partial
    # sums in the scratch array), F = 128; second call: a smaller matrix with
    # 300-entry rows and a ragged F = 37 (the generic path, whose long rows
    # are all split), leaving the first call's partials behind in the scratch
    if fmt in ("ell", "dia"):
        big = (4096, 4, 600, 20000)
        small = (1500, 2, 100, 6000)
    else:
        big = (20011, 6, 3000, 150000)
        small = (5003, 3, 300, 30000)
    for (R, hubs, hub_len, base), F, seed in ((big, 128, 11), (small, 37, 12)):
        row, col, val = _hub_matrix(R, hubs, hub_len, base, seed)
        X = graphgen.features_x(R, F, seed + 100)
        _check_pair(row, col, val, R, fmt, X, ldy_pad=5 if F == 37 else 0)


def test_noalloc_refuses_coo_and_oversized_workspace():
    R = 3000
    row, col, val = _hub_matrix(R, 1, 200, 9000, 21)
    d = (_dev(row), _dev(col), _dev(val))
    X = torch.ones((R, 16), dtype=torch.float32, device=DEV)
    Y = torch.empty((R, 16), dtype=torch.float32, device=DEV)
    m = gs.build_format(*d, (R, R), "coo")
    assert _noalloc(m, X, Y) == gs.ERR_UNSUPPORTED
    assert b"COO" in gs.lib().gs_last_error()
    m.close()
    # CSC needs 8 * R * F bytes: above the scratch for R = 70,000, F = 128
    R2 = 70_000
    r2, c2, v2 = graphgen.random_coo(R2, R2, 200_000, 22)
    m = gs.build_format(_dev(r2), _dev(c2), _dev(v2), (R2, R2), "csc")
    assert 8 * R2 * 128 > SCRATCH
    X2 = torch.ones((R2, 128), dtype=torch.float32, device=DEV)
    Y2 = torch.full((R2, 128), 3.0, dtype=torch.float32, device=DEV)
    assert _noalloc(m, X2, Y2) == gs.ERR_UNSUPPORTED
    assert b"scratch" in gs.lib().gs_last_error()
    torch.cuda.synchronize()
    assert (Y2 == 3.0).all(), "a refused call wrote Y"
    m.close()
