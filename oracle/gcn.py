"""Two-layer GCN training step in fp64 -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may use this module; it shares nothing with the GPU library.

The model is the two-layer graph convolution network of the paper's
motivating example (Sec. 3, after Kipf and Welling) and of its evaluation,
where two GNN layers are stacked (Sec. 5.1).  Each layer transforms the node
features with a dense weight and aggregates them over the graph with the
sparse adjacency (the SpMM of Sec. 2.1):

    Z1 = X W1,  P1 = A Z1,  H1 = relu(P1),  Z2 = H1 W2,  Out = A Z2,
    loss = sum((Out - T)^2) / (2 n)          (n = number of rows of A)

Backward, the chain rule written out (A^T is the transposed adjacency):

    G   = (Out - T) / n
    dZ2 = A^T G,     dW2 = H1^T dZ2,   dH1 = dZ2 W2^T,
    dP1 = dH1 * [P1 > 0],
    dZ1 = A^T dP1,   dW1 = X^T dZ1.

Everything is fp64: the aggregations use the oracle's fp64 SpMM on fp64
operands (``oracle.spmm64``), the dense products numpy fp64 matmul.
``magnitudes`` runs the same chain on |A|, |X|, |W|, |T| with no ReLU mask,
giving for every quantity an upper bound of the sum of absolute terms that
an fp32 evaluation rounds; the tests derive their tolerance from it.
"""
from __future__ import annotations

import numpy as np

import oracle


class Graph:
    """A and A^T in CSR (canonical order), from any COO triplets."""

    def __init__(self, R, C, row, col, val):
        self.R, self.C = int(R), int(C)
        r, c, v = oracle.canon(R, C, row, col, val)
        self.rp, self.col, self.val = oracle.csr(R, r), c, v
        rt, ct, vt = oracle.canon(C, R, col, row, val)
        self.rpT, self.colT, self.valT = oracle.csr(C, rt), ct, vt
        self.absval = np.abs(self.val)
        self.absvalT = np.abs(self.valT)

    def agg(self, Z, absolute=False):
        """A Z (fp64)."""
        return oracle.spmm64(self.R, self.rp, self.col, self.absval if absolute else self.val, Z)

    def agg_t(self, G, absolute=False):
        """A^T G (fp64)."""
        return oracle.spmm64(self.C, self.rpT, self.colT, self.absvalT if absolute else self.valT, G)


def forward_backward(g: Graph, X, W1, W2, T):
    """Forward values, loss and the gradients of the loss w.r.t. W1 and W2."""
    X, W1, W2, T = (np.asarray(a, dtype=np.float64) for a in (X, W1, W2, T))
    n = g.R
    Z1 = X @ W1
    P1 = g.agg(Z1)
    H1 = np.maximum(P1, 0.0)
    Z2 = H1 @ W2
    Out = g.agg(Z2)
    D = Out - T
    loss = float(np.sum(D * D)) / (2.0 * n)
    G = D / n
    dZ2 = g.agg_t(G)
    dW2 = H1.T @ dZ2
    dH1 = dZ2 @ W2.T
    dP1 = dH1 * (P1 > 0.0)
    dZ1 = g.agg_t(dP1)
    dW1 = X.T @ dZ1
    return dict(Z1=Z1, P1=P1, H1=H1, Z2=Z2, Out=Out, loss=loss, G=G, dZ2=dZ2, dW2=dW2,
                dH1=dH1, dP1=dP1, dZ1=dZ1, dW1=dW1)


def magnitudes(g: Graph, X, W1, W2, T):
    """The chain on absolute values without the ReLU mask: bounds the sum of
    absolute terms behind every quantity of ``forward_backward``."""
    X, W1, W2, T = (np.abs(np.asarray(a, dtype=np.float64)) for a in (X, W1, W2, T))
    n = g.R
    Z1 = X @ W1
    P1 = g.agg(Z1, absolute=True)
    Z2 = P1 @ W2
    Out = g.agg(Z2, absolute=True)
    G = (Out + T) / n
    dZ2 = g.agg_t(G, absolute=True)
    dW2 = P1.T @ dZ2
    dH1 = dZ2 @ W2.T
    dZ1 = g.agg_t(dH1, absolute=True)
    dW1 = X.T @ dZ1
    return dict(Z1=Z1, P1=P1, H1=P1, Z2=Z2, Out=Out, G=G, dZ2=dZ2, dW2=dW2, dH1=dH1, dP1=dH1,
                dZ1=dZ1, dW1=dW1)


def relu_ambiguity(g: Graph, X, ref, mag, eps, atol=0.0):
    """Extra bound on dW1 from ReLU decisions an fp32 evaluation may take the
    other way: entries of P1 within eps * |P1| + atol of zero (the error bound
    of the fp32 P1).  Flipping one such decision (i, h) changes dW1[:, h] by at
    most |dH1[i, h]| (|X|^T |A|^T e_i)."""
    amb = np.abs(ref["P1"]) <= eps * mag["P1"] + atol
    E = np.abs(mag["dH1"]) * amb
    extra = np.abs(np.asarray(X, dtype=np.float64)).T @ g.agg_t(E, absolute=True)
    return extra, int(amb.sum())


def sgd_step(W1, W2, grads, lr):
    return W1 - lr * grads["dW1"], W2 - lr * grads["dW2"]
