"""Operands past the int32 range of elements.

R = C = 2^23 + 2^20 + 37 and F = 256, so X and Y hold 2.4e9 elements each:
the gather offsets j * ldx of the top 2^20 columns, the stores row * ldy of
the top 2^20 rows and the CSC workspace index row * F all exceed 2^31.  The
header allows n_rows, n_cols and nnz below 2^31 with 64-bit F and strides.

The matrix is a band (offsets -2, 0, 3) plus a far diagonal, so every format
is feasible.  X repeats a seeded base of P = 4099 rows (a prime, so no
multiple of 2^32 elements maps a row onto an equal one).  Y is pre-filled
with NaN, so a row left unwritten fails; sampled rows (first and last, both
sides of row 2^23 and of the far diagonal's switch, and a seeded sample) are
checked against the oracle, which receives the sampled rows and the X rows
they touch."""
import numpy as np
import pytest
import torch

import graphgen
import oracle
import paper_2111_00352_amd as gs

pytestmark = pytest.mark.gpu

N = (1 << 23) + (1 << 20) + 37
F = 256
P = 4099
FMTS = ["csr", "coo", "ell", "dia", "bsr", "csc"]


@pytest.fixture(scope="module")
def big():
    row, col, val = graphgen.band_far_coo(N, seed=4242)
    base = graphgen.features_x(P, F, seed=4243)
    rp = oracle.csr(N, row)
    rng = np.random.default_rng(4244)
    pick = [0, 1, 2, N - 3, N - 2, N - 1, (1 << 23) - 1, 1 << 23, (1 << 23) + 1,
            N - N // 2 - 1, N - N // 2]
    pick += list(rng.choice(N, size=300, replace=False))
    rows = np.unique(np.array(pick, dtype=np.int64))
    # the sampled rows as a small CSR over the X rows they touch
    seg = [np.arange(rp[r], rp[r + 1]) for r in rows]
    idx = np.concatenate(seg)
    sub_rp = np.concatenate([[0], np.cumsum([s.size for s in seg])]).astype(np.int32)
    cols, sub_col = np.unique(col[idx], return_inverse=True)
    Yref, M = oracle.spmm_rows(np.arange(rows.size), sub_rp, sub_col.astype(np.int32), val[idx],
                               base[cols % P])
    dev = "cuda"
    X = torch.from_numpy(base).to(dev)[torch.arange(N, device=dev) % P]
    assert X.is_contiguous() and X.numel() > (1 << 31)
    return dict(row=torch.from_numpy(row).to(dev), col=torch.from_numpy(col).to(dev),
                val=torch.from_numpy(val).to(dev), X=X, rows=rows, Yref=Yref, M=M)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("fmt", FMTS)
def test_offsets_past_int32(big, fmt):
    m = gs.build_format(big["row"], big["col"], big["val"], (N, N), fmt)
    Y = torch.full((N, F), float("nan"), device="cuda")
    m.spmm(big["X"], out=Y)
    assert not bool(torch.isnan(Y).any()), f"{fmt}: rows left unwritten"
    Yh = Y[torch.from_numpy(big["rows"]).cuda()].cpu().numpy()
    ok, worst = oracle.check_spmm(Yh, big["Yref"], big["M"])
    assert ok, f"{fmt}: worst |err|/bound {worst}"
    m.close()
    del Y
    torch.cuda.empty_cache()



# The largest entry count the header allows: 2^27 - 5 rows with 16 band
# entries each (edges clipped), 2^31 - 329 entries.  Entry indices, row
# pointers, range bounds, radix-sort positions and the CSC permutation then
# run up to the top of the int32 range; ELL's K*R slots and DIA's data pass
# 2^31.  The padded formats exceed the default 8 GiB cap at this size, so
# ELL and DIA are built under a 40 GiB cap (BSR would need about 60 GB).
NZ_ROWS = (1 << 27) - 5
NZ_OFFS = np.array([-7, -5, -3, -2, -1, 0, 1, 2, 3, 5, 8, 13, 21, 34, 55, 89], np.int32)


@pytest.fixture(scope="module")
def most_entries():
    n = NZ_ROWS
    row = np.repeat(np.arange(n, dtype=np.int32), NZ_OFFS.size)
    col = row + np.tile(NZ_OFFS, n)
    keep = (col >= 0) & (col < n)
    row, col = row[keep], col[keep]
    del keep
    assert row.size == (1 << 31) - 329
    # values k/2^16 + 1/2 for k = entry index mod 2^16: exact, never zero
    val = (np.arange(row.size, dtype=np.uint32) & 0xFFFF).astype(np.float32) * np.float32(2.0**-16)
    val += np.float32(0.5)
    X = graphgen.features_x(n, 4, seed=4245)
    rng = np.random.default_rng(4246)
    pick = [0, 1, 7, 88, 89, n // 2, n - 90, n - 89, n - 8, n - 1]
    pick += list(rng.choice(n, size=200, replace=False))
    rows = np.unique(np.array(pick, dtype=np.int64))
    starts = np.searchsorted(row, rows)
    ends = np.searchsorted(row, rows, side="right")
    seg = [np.arange(s, e) for s, e in zip(starts, ends)]
    idx = np.concatenate(seg)
    sub_rp = np.concatenate([[0], np.cumsum([s.size for s in seg])]).astype(np.int32)
    cols, sub_col = np.unique(col[idx], return_inverse=True)
    Yref, M = oracle.spmm_rows(np.arange(rows.size), sub_rp, sub_col.astype(np.int32), val[idx], X[cols])
    dev = "cuda"
    out = dict(row=torch.from_numpy(row).to(dev), col=torch.from_numpy(col).to(dev),
               val=torch.from_numpy(val).to(dev), X=torch.from_numpy(X).to(dev), rows=rows, Yref=Yref, M=M)
    del row, col, val
    return out


@pytest.mark.timeout(600)
@pytest.mark.parametrize("fmt", ["csr", "coo", "csc", "ell", "dia"])
def test_most_entries(most_entries, fmt):
    b = most_entries
    m = gs.build_format(b["row"], b["col"], b["val"], (NZ_ROWS, NZ_ROWS), fmt, max_bytes=40 << 30)
    Y = torch.full((NZ_ROWS, 4), float("nan"), device="cuda")
    m.spmm(b["X"], out=Y)
    assert not bool(torch.isnan(Y).any()), f"{fmt}: rows left unwritten"
    Yh = Y[torch.from_numpy(b["rows"]).cuda()].cpu().numpy()
    del Y
    ok, worst = oracle.check_spmm(Yh, b["Yref"], b["M"])
    assert ok, f"{fmt}: worst |err|/bound {worst}"
    if fmt in ("ell", "dia"):  # the padded layouts give back the canonical COO, bit for bit
        r, c, v = m.to_coo()
        assert torch.equal(r, b["row"]) and torch.equal(c, b["col"])
        assert torch.equal(v.view(torch.int32), b["val"].view(torch.int32))
        del r, c, v
    m.close()
    torch.cuda.empty_cache()


def _band_aggregates(n, offs):
    """Integer aggregates of the n x n matrix with entries (i, i+o), o in offs,
    worked out from the band's geometry: every row and column away from the
    edges holds len(offs) entries, and the 16x16 block pattern of a block row
    repeats along the band, so only the first and last rows and block rows
    are enumerated."""
    offs = [int(o) for o in offs]
    k = len(offs)
    edge = max(abs(o) for o in offs) + 1
    assert n > 2 * edge  # every offset then has entries, and the ends do not meet

    def counts(sign):  # entries of line i: offsets with 0 <= i + sign*o < n
        idx = list(range(min(edge, n))) + list(range(max(edge, n - edge), n))
        c = {i: sum(1 for o in offs if 0 <= i + sign * o < n) for i in idx}
        interior = n - len(c)
        s2 = sum(v * v for v in c.values()) + interior * k * k
        full = [c.get(i, k) for i in range(min(edge + 1, n))] + [c.get(i, k) for i in range(max(edge + 1, n - edge - 1), n)]
        bounce = sum(abs(full[j + 1] - full[j]) for j in range(len(full) - 1))
        return max(c.values()), min(c.values()), s2, bounce

    max_r, min_r, s2r, br = counts(+1)
    max_c, min_c, s2c, bc = counts(-1)
    nbr = (n + 15) // 16
    eb = edge // 16 + 2

    def blocks(b):
        ds = set()
        for kk in range(16):
            i = 16 * b + kk
            if i >= n:
                break
            for o in offs:
                if 0 <= i + o < n:
                    ds.add((i + o) // 16)
        return len(ds)

    ends = sorted(set(range(min(eb, nbr))) | set(range(max(0, nbr - eb), nbr)))
    nb16 = sum(blocks(b) for b in ends) + (nbr - len(ends)) * blocks(nbr // 2)
    return {"n_rows": n, "n_cols": n, "n_diags": k, "max_rd": max_r, "min_rd": min_r, "max_cd": max_c,
            "min_cd": min_c, "sum_rd2": s2r, "sum_cd2": s2c, "bounce_r": br, "bounce_c": bc,
            "n_blocks16": nb16}


def test_band_aggregates_match_the_oracle_on_a_small_band():
    # the closed forms above, checked against the oracle where it is fast
    n = 1000
    row = np.repeat(np.arange(n, dtype=np.int32), NZ_OFFS.size)
    col = row + np.tile(NZ_OFFS, n)
    keep = (col >= 0) & (col < n)
    ints, _ = oracle.features(n, n, row[keep], col[keep])
    exp = _band_aggregates(n, NZ_OFFS)
    exp["nnz"] = int(keep.sum())
    assert ints == exp


@pytest.mark.timeout(600)
def test_features_at_most_entries(most_entries):
    b = most_entries
    got = gs.extract_features(b["row"], b["col"], b["val"], (NZ_ROWS, NZ_ROWS))
    exp = _band_aggregates(NZ_ROWS, NZ_OFFS)
    exp["nnz"] = (1 << 31) - 329
    assert {k: got[k] for k in exp} == exp
