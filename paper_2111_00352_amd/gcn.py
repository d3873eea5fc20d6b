"""Two-layer GCN training with the selector deciding each aggregation's format.

The paper's end-to-end setting (Sec. 3 motivating example, Sec. 5.1-5.2): a
two-layer graph convolution network trained for a number of epochs, where
every aggregation is an SpMM whose storage format the predictor chooses once
per layer and reuses across epochs (Sec. 4.6).  Per layer

    forward:   Y = A . (H W)           (aggregation of transformed features)
    backward:  d(HW) = A^T . dY        (the aggregation of the gradient)

Both aggregations go through ``SelectContext.run`` (features extracted once
per adjacency key, the format predicted per call since the feature width F is
one of the predictor's inputs, converted at most once per key).  A^T is a
second key built from the same triplets with rows and columns exchanged, or
the same key when the caller declares A symmetric (GCN-normalised adjacencies
are).  The dense products H W and their gradients are PyTorch fp32 matmuls
(the weight gradient H^T G, an n-long reduction, split over row chunks);
ReLU and the loss are PyTorch element-wise operations.

Command line (end-to-end timing of one workload):
    python -m paper_2111_00352_amd.gcn --config 2 --epochs 10
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import torch

from paper_2111_00352_amd import SelectContext


class Adjacency:
    """A (and A^T) as COO triplets on the device, aggregated through a selector."""

    def __init__(self, row, col, val, shape, ctx: SelectContext, key: int, symmetric: bool = False):
        self.row, self.col, self.val = row, col, val
        self.R, self.C = int(shape[0]), int(shape[1])
        self.ctx = ctx
        self.key = int(key)
        self.symmetric = bool(symmetric) and self.R == self.C
        self.key_t = self.key if self.symmetric else self.key + 1
        self.chosen = []  # (key, F, format) of every aggregation, in call order

    def agg(self, Z: torch.Tensor) -> torch.Tensor:
        Y, fmt = self.ctx.run(self.key, self.row, self.col, self.val, (self.R, self.C), Z)
        self.chosen.append((self.key, Z.shape[1], fmt))
        return Y

    def agg_t(self, G: torch.Tensor) -> torch.Tensor:
        if self.symmetric:
            Y, fmt = self.ctx.run(self.key, self.row, self.col, self.val, (self.R, self.C), G)
        else:
            Y, fmt = self.ctx.run(self.key_t, self.col, self.row, self.val, (self.C, self.R), G)
        self.chosen.append((self.key_t, G.shape[1], fmt))
        return Y


class _Aggregate(torch.autograd.Function):
    @staticmethod
    def forward(ctx, Z, adj):
        ctx.adj = adj
        return adj.agg(Z.contiguous())

    @staticmethod
    def backward(ctx, dY):
        return ctx.adj.agg_t(dY.contiguous()), None


def aggregate(Z: torch.Tensor, adj: Adjacency) -> torch.Tensor:
    return _Aggregate.apply(Z, adj)


def weight_grad(H: torch.Tensor, G: torch.Tensor, rows_per_chunk: int = 2048) -> torch.Tensor:
    """H^T G for tall H (n x a) and G (n x b): the n-long reduction is split
    over row chunks (one batched product, then a sum over the chunks), which
    keeps the GPU busy where a single a x b product with an n-long inner
    dimension would not."""
    n = H.shape[0]
    k = n // rows_per_chunk
    if k < 2:
        return H.t() @ G
    m = n // k
    main = k * m
    Hc = H[:main].reshape(k, m, H.shape[1]).transpose(1, 2).contiguous()
    Gc = G[:main].reshape(k, m, G.shape[1])
    out = torch.bmm(Hc, Gc).sum(0)
    if main < n:
        out = out + H[main:].t() @ G[main:]
    return out


class _Linear(torch.autograd.Function):
    """H W with the weight gradient formed by ``weight_grad``."""

    @staticmethod
    def forward(ctx, H, W):
        ctx.save_for_backward(H, W)
        return H @ W

    @staticmethod
    def backward(ctx, G):
        H, W = ctx.saved_tensors
        G = G.contiguous()
        dH = G @ W.t() if ctx.needs_input_grad[0] else None
        dW = weight_grad(H, G) if ctx.needs_input_grad[1] else None
        return dH, dW


class GCN2:
    """Weights of the two layers (fp32, on the device); forward and SGD step."""

    def __init__(self, W1: torch.Tensor, W2: torch.Tensor):
        self.W1 = W1.detach().clone().requires_grad_(True)
        self.W2 = W2.detach().clone().requires_grad_(True)

    def forward(self, X, adj: Adjacency):
        P1 = aggregate(_Linear.apply(X, self.W1), adj)
        H1 = torch.relu(P1)
        return aggregate(_Linear.apply(H1, self.W2), adj), P1

    def loss(self, Out, T):
        return ((Out - T) ** 2).sum() / (2.0 * Out.shape[0])

    def step(self, X, T, adj: Adjacency, lr: float):
        """One training step; returns (loss, Out, P1) with the gradients in
        W1.grad / W2.grad and the weights updated by SGD."""
        self.W1.grad = None
        self.W2.grad = None
        Out, P1 = self.forward(X, adj)
        loss = self.loss(Out, T)
        loss.backward()
        with torch.no_grad():
            self.W1 -= lr * self.W1.grad
            self.W2 -= lr * self.W2.grad
        return loss.detach(), Out.detach(), P1.detach()


def train(adj: Adjacency, X, T, W1, W2, epochs: int, lr: float, graph: bool = False):
    """Trains for `epochs` steps; returns (model, per-epoch losses, seconds per epoch).

    graph=True: the first two epochs run eagerly (format selection, conversion
    and workspace growth happen there, and the second runs on a side stream
    as the capture recipe asks), then one training step is captured into a
    HIP graph and replayed for the remaining epochs.  The format choice is
    frozen in the graph, as the paper decides it once per layer across
    epochs (Sec. 5.2); every SpMM path launches kernels only once warm (no
    allocation, memset or synchronisation), so it records cleanly."""
    model = GCN2(W1, W2)
    losses, times = [], []
    eager = epochs if not graph else min(epochs, 2)
    for e in range(eager):
        t0 = time.perf_counter()
        if graph and e == eager - 1:
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                loss, _, _ = model.step(X, T, adj, lr)
            torch.cuda.current_stream().wait_stream(side)
        else:
            loss, _, _ = model.step(X, T, adj, lr)
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
        losses.append(float(loss))
    if epochs > eager:
        t0 = time.perf_counter()
        g = torch.cuda.CUDAGraph()
        model.W1.grad = None
        model.W2.grad = None
        with torch.cuda.graph(g):
            static_loss, _, _ = model.step(X, T, adj, lr)
        for e in range(eager, epochs):
            g.replay()
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
            losses.append(float(static_loss))
            t0 = time.perf_counter()
    return model, losses, times


def end_to_end(row, col, val, shape, X, T, W1, W2, epochs=10, lr=0.1, symmetric=False,
               modes=("model", "fixed:csr", "fixed:coo"), graph=False, passes=2):
    """Trains once per selection mode, each with a fresh context (so every
    first-call cost -- features, prediction, conversion -- is paid inside the
    timed epochs), and reports total time and the speedups of the first mode
    over the others (Sec. 5.2: end-to-end time over 10 epochs, overheads
    included).  The modes are timed in turn `passes` times and the last pass
    is reported: whichever mode is timed first in a process runs its epochs
    some 3% slower (measured with the modes in every order), which would
    otherwise be charged to the first mode."""
    # untimed epochs first, once per mode, each in a context of its own:
    # PyTorch's GEMM and autograd start-up and the first launch of each
    # format's kernels happen once per process, not per matrix
    for mode in modes:
        name, _, fixed = mode.partition(":")
        warm = SelectContext(name, fixed=fixed or "csr")
        train(Adjacency(row, col, val, shape, warm, key=1, symmetric=symmetric), X, T, W1, W2,
              3 if graph else 1, lr, graph=graph)
        warm.close()
    res = {}
    for _ in range(max(1, passes)):
        for mode in modes:
            name, _, fixed = mode.partition(":")
            ctx = SelectContext(name, fixed=fixed or "csr")
            adj = Adjacency(row, col, val, shape, ctx, key=7, symmetric=symmetric)
            torch.cuda.synchronize()
            _, losses, times = train(adj, X, T, W1, W2, epochs, lr, graph=graph)
            res[mode] = {
                "total_s": sum(times), "first_epoch_s": times[0],
                "steady_epoch_s": sorted(times[1:])[len(times[1:]) // 2] if len(times) > 1 else times[0],
                "final_loss": losses[-1],
                "formats": sorted({f"key{k}/F{F}:{fmt}" for k, F, fmt in adj.chosen}),
            }
            ctx.close()
    base = modes[0]
    for m in modes[1:]:
        res[f"speedup_{base}_vs_{m}"] = res[m]["total_s"] / res[base]["total_s"]
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--epochs", type=int, default=10)
    ap.add_argument("--hidden", type=int, default=128)
    ap.add_argument("--out", type=int, default=64)
    ap.add_argument("--lr", type=float, default=0.02)
    ap.add_argument("--graph", action="store_true", help="replay a captured training step after two epochs")
    a = ap.parse_args()
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import graphgen

    torch.backends.cuda.matmul.allow_tf32 = False
    g = graphgen.config(a.config)
    dev = torch.device("cuda", 0)
    row, col, val = (torch.from_numpy(x).to(dev) for x in (g.row, g.col, g.val))
    X = torch.from_numpy(g.X).to(dev)
    W1 = torch.from_numpy(graphgen.features_x(g.F, a.hidden, 4100 + a.config, "normal")).to(dev) / g.F ** 0.5
    W2 = torch.from_numpy(graphgen.features_x(a.hidden, a.out, 4200 + a.config, "normal")).to(dev) / a.hidden ** 0.5
    T = torch.from_numpy(graphgen.features_x(g.R, a.out, 4300 + a.config, "normal")).to(dev)
    res = end_to_end(row, col, val, (g.R, g.C), X, T, W1, W2, a.epochs, a.lr,
                     symmetric=bool(g.meta.get("symmetric", False)), graph=a.graph)
    print(json.dumps({"workload": g.name, "epochs": a.epochs, "hidden": a.hidden, "out": a.out,
                      "graph": a.graph, **res}))


if __name__ == "__main__":
    main()
