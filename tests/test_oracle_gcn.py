"""Pins of the fp64 two-layer GCN oracle (oracle/gcn.py) against mathematics
it does not itself use: dense brute force for the forward values and the
transposed aggregation, central finite differences of the loss for the
gradients, and the magnitude pass bounding every value."""
import numpy as np
import pytest

import graphgen
from oracle import gcn


def _problem(n=11, C=None, F=3, H=4, O=2, nnz=30, seed=5, empty=0.2):
    C = n if C is None else C
    row, col, val = graphgen.random_coo(n, C, nnz, seed, empty_rows=empty)
    rng = np.random.default_rng(seed + 1)
    X = rng.standard_normal((C, F))
    W1 = rng.standard_normal((F, H))
    W2 = rng.standard_normal((H, O))
    T = rng.standard_normal((n, O))
    return gcn.Graph(n, C, row, col, val), (row, col, val), X, W1, W2, T


def _dense(n, C, row, col, val):
    A = np.zeros((n, C))
    A[row, col] = val.astype(np.float64)
    return A


def test_forward_matches_dense_brute_force():
    # square (the GCN case) and rectangular aggregations, with empty rows
    for n, C in ((11, 11), (13, 7)):
        g, (row, col, val), X, W1, W2, T = _problem(n=n, C=C, nnz=35)
        A = _dense(n, C, row, col, val)
        if n == C:
            ref = gcn.forward_backward(g, X, W1, W2, T)
            P1 = A @ (X @ W1)
            Out = A @ (np.maximum(P1, 0) @ W2)
            assert np.allclose(ref["P1"], P1, rtol=1e-13, atol=1e-13)
            assert np.allclose(ref["Out"], Out, rtol=1e-13, atol=1e-13)
            assert ref["loss"] == pytest.approx(np.sum((Out - T) ** 2) / (2 * n), rel=1e-13)
        Y = np.random.default_rng(9).standard_normal((n, 5))
        assert np.allclose(g.agg_t(Y), A.T @ Y, rtol=1e-13, atol=1e-13)
        Z = np.random.default_rng(10).standard_normal((C, 5))
        assert np.allclose(g.agg(Z), A @ Z, rtol=1e-13, atol=1e-13)


def _fd_check(g, X, W1, W2, T, h=1e-6):
    ref = gcn.forward_backward(g, X, W1, W2, T)
    # rows of A with no entries give exact zeros that stay zero under any
    # perturbation of W; every other ReLU input must be away from the kink
    P1 = ref["P1"][ref["P1"] != 0]
    assert np.min(np.abs(P1)) > 1e-3, "a ReLU input sits on the kink"
    worst = 0.0
    for name, W in (("dW1", W1), ("dW2", W2)):
        for idx in np.ndindex(W.shape):
            Wp, Wm = W.copy(), W.copy()
            Wp[idx] += h
            Wm[idx] -= h
            args_p = (Wp, W2) if name == "dW1" else (W1, Wp)
            args_m = (Wm, W2) if name == "dW1" else (W1, Wm)
            lp = gcn.forward_backward(g, X, *args_p, T)["loss"]
            lm = gcn.forward_backward(g, X, *args_m, T)["loss"]
            fd = (lp - lm) / (2 * h)
            an = ref[name][idx]
            worst = max(worst, abs(fd - an) / (abs(an) + 1e-6))
    return worst


@pytest.mark.parametrize("n,C,seed", [(11, 11, 5), (17, 17, 6)])
def test_gradients_match_finite_differences(n, C, seed):
    g, _, X, W1, W2, T = _problem(n=n, C=C, nnz=3 * n, seed=seed)
    assert _fd_check(g, X, W1, W2, T) < 1e-6


def test_planted_transpose_mistake_is_caught(monkeypatch):
    # aggregating the backward with A instead of A^T (a non-symmetric A) must
    # fail the finite-difference pin
    g, _, X, W1, W2, T = _problem(n=11, nnz=33, seed=5)
    monkeypatch.setattr(gcn.Graph, "agg_t", lambda self, G, absolute=False: self.agg(G, absolute))
    assert _fd_check(g, X, W1, W2, T) > 1e-2


def test_magnitudes_bound_every_value():
    g, _, X, W1, W2, T = _problem(n=40, nnz=160, seed=8)
    ref = gcn.forward_backward(g, X, W1, W2, T)
    mag = gcn.magnitudes(g, X, W1, W2, T)
    for k, v in mag.items():
        assert np.all(np.abs(ref[k]) <= v * (1 + 1e-12) + 1e-300), k


def test_relu_ambiguity_bound_covers_a_flipped_decision():
    # flip the smallest ReLU decision by hand: the change in dW1 stays within
    # the ambiguity bound computed with an eps that makes that entry ambiguous
    g, _, X, W1, W2, T = _problem(n=30, nnz=120, seed=12)
    ref = gcn.forward_backward(g, X, W1, W2, T)
    mag = gcn.magnitudes(g, X, W1, W2, T)
    r = np.full(mag["P1"].shape, np.inf)
    np.divide(np.abs(ref["P1"]), mag["P1"], out=r, where=mag["P1"] > 0)
    i, h = np.unravel_index(np.argmin(r), r.shape)
    mask = ref["P1"] > 0
    mask[i, h] = not mask[i, h]
    dW1_flipped = X.T @ g.agg_t(ref["dH1"] * mask)
    extra, count = gcn.relu_ambiguity(g, X, ref, mag, eps=r[i, h] * 1.0001)
    assert count >= 1
    assert np.all(np.abs(dW1_flipped - ref["dW1"]) <= extra * (1 + 1e-9) + 1e-15)


def _atol_branch_holds(relu_ambiguity):
    """The absolute term of the ambiguity test (atol, the 1e-6 absolute part
    of the SpMM bound) on its own: with eps = 0 the ReLU input of smallest
    magnitude is ambiguous exactly when atol reaches |P1[i, h]|, and the
    bound then covers flipping that decision."""
    g, _, X, W1, W2, T = _problem(n=30, nnz=120, seed=14)
    ref = gcn.forward_backward(g, X, W1, W2, T)
    mag = gcn.magnitudes(g, X, W1, W2, T)
    a = np.abs(ref["P1"])
    a[mag["P1"] == 0] = np.inf  # exact zeros of empty rows are never ambiguous in the check
    i, h = np.unravel_index(np.argmin(a), a.shape)
    p = a[i, h]
    mask = ref["P1"] > 0
    mask[i, h] = not mask[i, h]
    dW1_flipped = X.T @ g.agg_t(ref["dH1"] * mask)
    extra, count = relu_ambiguity(g, X, ref, mag, eps=0.0, atol=p * 1.0001)
    _, count_below = relu_ambiguity(g, X, ref, mag, eps=0.0, atol=p * 0.9999)
    covered = np.all(np.abs(dW1_flipped - ref["dW1"]) <= extra * (1 + 1e-9) + 1e-15)
    return count >= 1 and count_below == count - 1 and bool(covered)


def test_relu_ambiguity_absolute_term():
    assert _atol_branch_holds(gcn.relu_ambiguity)


def test_relu_ambiguity_planted_sign_mistake_is_caught():
    # the absolute term subtracted instead of added: the entry within atol of
    # zero is no longer ambiguous, and the bound misses its flip
    def planted(g, X, ref, mag, eps, atol=0.0):
        amb = np.abs(ref["P1"]) <= eps * mag["P1"] - atol
        E = np.abs(mag["dH1"]) * amb
        return np.abs(np.asarray(X, dtype=np.float64)).T @ g.agg_t(E, absolute=True), int(amb.sum())

    assert not _atol_branch_holds(planted)
