"""Full-size parity: every workload at its real shape, through the selector
(the launch configuration the benchmark times) and through every feasible
format.  Every element of Y is checked against the oracle's full fp64
result (|Y - Y_ref| <= 1e-5 (|A||X|) + 1e-6), every feasible format's arrays
are compared with the oracle's canonical layout byte for byte, and the
features must be exact.

The large workload's second layer takes ReLU((A X1) W) as input, built on the
CPU from the oracle's own first-layer output."""
import numpy as np
import pytest
import torch

import graphgen
import oracle
import paper_2111_00352_amd as gs

pytestmark = pytest.mark.gpu

FMTS = ["csr", "coo", "ell", "dia", "bsr", "csc"]
CHUNK = 1 << 16  # rows per comparison step


class Full:
    def __init__(self, k):
        g = graphgen.config(k)
        self.g = g
        self.rp = oracle.csr(g.R, g.row)
        dev = "cuda"
        self.row, self.col, self.val = (torch.from_numpy(a).to(dev) for a in (g.row, g.col, g.val))
        self.X = torch.from_numpy(g.X).to(dev)
        self._ref = None

    def ref(self):
        """The oracle's whole Y (fp64) and |A||X| for X."""
        if self._ref is None:
            self._ref = oracle.spmm(self.g.R, self.rp, self.g.col, self.g.val, self.g.X)
        return self._ref

    def check(self, Y, ref=None, label=""):
        """Every element of Y [dev] against the oracle, a block of rows at a time."""
        Yref, M = self.ref() if ref is None else ref
        worst = 0.0
        for r0 in range(0, self.g.R, CHUNK):
            r1 = min(self.g.R, r0 + CHUNK)
            ok, w = oracle.check_spmm(Y[r0:r1].cpu().numpy(), Yref[r0:r1], M[r0:r1])
            assert ok, f"{label}: rows {r0}..{r1}: worst |err|/bound {w}"
            worst = max(worst, w)
        return worst

    def layout(self, fmt, b=16):
        """The oracle's canonical arrays of format fmt."""
        g = self.g
        if fmt == "csr":
            return [self.rp, g.col, g.val]
        if fmt == "coo":
            return [g.row, g.col, g.val]
        if fmt == "csc":
            return list(oracle.csc(g.R, g.C, g.row, g.col, g.val))
        if fmt == "ell":
            return list(oracle.ell(g.R, self.rp, g.col, g.val)[1:])
        if fmt == "dia":
            return list(oracle.dia(g.R, g.C, g.row, g.col, g.val))
        return list(oracle.bsr(g.R, g.C, b, g.row, g.col, g.val))


_cache = {}


def full(k):
    if k not in _cache:
        _cache.clear()
        _cache[k] = Full(k)
    return _cache[k]


def _same_bytes(got, exp):
    exp = np.ascontiguousarray(exp).astype(got.dtype, copy=False)
    return got.size == exp.size and (got.view(np.uint32) == exp.view(np.uint32)).all()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_fullsize_selector_and_features(k):
    f = full(k)
    g = f.g
    ctx = gs.SelectContext("model")
    Y, fmt = ctx.run(1, f.row, f.col, f.val, (g.R, g.C), f.X)
    Y, fmt2 = ctx.run(1, f.row, f.col, f.val, (g.R, g.C), f.X)  # steady state (cached)
    assert fmt == fmt2
    f.check(Y, label=f"selector/{fmt}")
    ints, feats = oracle.features(g.R, g.C, g.row, g.col)
    got = gs.extract_features(f.row, f.col, f.val, (g.R, g.C))
    assert all(got[n] == v for n, v in ints.items())
    assert got["f"] == feats.tolist()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_fullsize_every_feasible_format(k):
    f = full(k)
    g = f.g
    for fmt in FMTS:
        try:
            m = gs.build_format(f.row, f.col, f.val, (g.R, g.C), fmt)
        except gs.GnnSpmmError as e:
            assert e.code == gs.ERR_INFEASIBLE, str(e)
            continue
        f.check(m.spmm(f.X), label=fmt)
        exp = f.layout(fmt)
        for which, e in enumerate(exp):  # canonical arrays, byte for byte
            got = m.array(which).cpu().numpy()
            assert _same_bytes(got, e), f"{fmt}: array {which}"
            del got
        if fmt in ("ell", "dia", "bsr"):
            assert m.param == (exp[0].size if fmt == "dia" else exp[1].size if fmt == "bsr" else exp[0].size // g.R)
        del exp
        m.close()
        torch.cuda.empty_cache()


@pytest.mark.timeout(600)
def test_fullsize_large_two_layers():
    # layer 2 re-selects on the same adjacency (cache hit) with the ReLU output
    f = full(5)
    g = f.g
    Y1ref, _ = f.ref()
    W = graphgen.layer2_weight(g.F)
    X2 = np.maximum(Y1ref.astype(np.float32) @ W, 0.0).astype(np.float32)
    assert 0.3 < float((X2 == 0).mean()) < 0.7  # about half zeros, as specified
    ctx = gs.SelectContext("model")
    Y1, fmt1 = ctx.run(5, f.row, f.col, f.val, (g.R, g.C), f.X)
    f.check(Y1, label=f"layer1/{fmt1}")
    X2d = torch.from_numpy(X2).cuda()
    Y2, fmt2 = ctx.run(5, f.row, f.col, f.val, (g.R, g.C), X2d)
    assert ctx.stats()["t_convert"] >= 0
    ref2 = oracle.spmm(g.R, f.rp, g.col, g.val, X2)
    f.check(Y2, ref=ref2, label=f"layer2/{fmt2}")
