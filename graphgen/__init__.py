"""Seeded synthetic inputs for the GNN aggregation SpMM.

This module holds only input generation: graph structure, edge values and the
dense feature matrix X.  It contains none of the SpMM, format-conversion or
feature arithmetic, and it is used by both the oracle tests and the GPU tests
and benchmark.

Randomness: numpy's ``Generator(PCG64(seed))`` (O'Neill 2014).  Value recipes
use integer draws scaled by powers of two so every fp32 value is exact:

* uniform (0,1)  : (k + 0.5) * 2^-24,   k uniform in [0, 2^24)
* uniform (0,1]  : (2^24 - k) * 2^-24
* uniform [-1,1) : k * 2^-23 - 1
* N(0,1)         : numpy's standard normal in fp64, rounded to fp32

Workloads (the paper measures on real graph suites and on small random 0/1
matrices; these synthetic, GNN-shaped graphs stand in for them):

1. ``tiny``: Erdos-Renyi G(n, p=4/(n-1)), n=2048, one Bernoulli draw per
   unordered pair; symmetrised, self-loops, GCN values D^-1/2 (A+I) D^-1/2;
   X n x 64 uniform[-1,1).
2. ``powerlaw``: Chung-Lu, n=100,000, exponent 2.1, mean degree 10, expected
   degree capped at 5,000; symmetrised, self-loops, GCN values; X n x 128 N(0,1).
3. ``mesh``: 512 x 512 grid, 5-point stencil incl. the centre, row-major ids,
   non-periodic (5 diagonals); values uniform(0,1], not symmetric;
   X n x 64 uniform[-1,1).
4. ``blocks``: n=204,800 in 12,800 contiguous communities of 16; Bernoulli(0.8)
   per unordered intra pair; 2 uniformly drawn partners per node outside its
   community; symmetrised, self-loops, GCN values; X n x 256 N(0,1).
5. ``large``: Chung-Lu, n=2,000,000, exponent 2.0, mean degree 25, cap
   floor(sqrt(25 n)) = 7071; symmetrised, self-loops; values uniform(0,1) per
   entry divided by their row sum (row-stochastic); X n x 128 N(0,1).  The
   second layer's input is ReLU((A X) W) with W 128x128 N(0, 1/128), computed
   by the caller.

Every graph is returned as canonical COO: sorted by (row, col), no duplicate
coordinates, no stored zeros.
"""
from __future__ import annotations

import dataclasses
import functools
import math

import numpy as np

__all__ = ["Graph", "config", "scaled", "CONFIG_NAMES", "random_coo", "shuffled", "features_x"]


@dataclasses.dataclass
class Graph:
    name: str
    R: int
    C: int
    row: np.ndarray  # int32, canonical order
    col: np.ndarray  # int32
    val: np.ndarray  # float32
    X: np.ndarray    # float32 C x F, row-major
    meta: dict

    @property
    def nnz(self) -> int:
        return int(self.row.size)

    @property
    def F(self) -> int:
        return int(self.X.shape[1])


CONFIG_NAMES = {1: "tiny", 2: "powerlaw", 3: "mesh", 4: "blocks", 5: "large"}


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _u01_open(rng, n):
    return ((rng.integers(0, 1 << 24, size=n, dtype=np.int64) + 0.5) * 2.0**-24).astype(np.float32)


def _u01_closed_top(rng, n):
    return (((1 << 24) - rng.integers(0, 1 << 24, size=n, dtype=np.int64)) * 2.0**-24).astype(np.float32)


def _um11(rng, shape):
    k = rng.integers(0, 1 << 24, size=shape, dtype=np.int64)
    return (k * 2.0**-23 - 1.0).astype(np.float32)


def _normal(rng, shape):
    return rng.standard_normal(size=shape).astype(np.float32)


def _canon_from_keys(keys: np.ndarray, n_cols: int):
    keys = np.unique(keys)
    row = (keys // n_cols).astype(np.int32)
    col = (keys % n_cols).astype(np.int32)
    return row, col


def _sym_with_self(u: np.ndarray, v: np.ndarray, n: int):
    """Union of (u,v), (v,u) and the n self-loops, deduplicated, sorted."""
    u = u.astype(np.int64)
    v = v.astype(np.int64)
    diag = np.arange(n, dtype=np.int64)
    keys = np.concatenate([u * n + v, v * n + u, diag * n + diag])
    return _canon_from_keys(keys, n)


def _gcn_values(row, col, n):
    deg = np.bincount(row, minlength=n).astype(np.float64)
    return (1.0 / np.sqrt(deg[row] * deg[col])).astype(np.float32)


def _erdos_renyi_pairs(rng, n, p):
    iu, ju = np.triu_indices(n, k=1)
    keep = rng.random(iu.size) < p
    return iu[keep], ju[keep]


def _chung_lu_pairs(rng, n, gamma, mean_deg, cap):
    """Chung-Lu by edge sampling.  Expected degree w_i = min(cap, s (i+1)^(-1/(gamma-1)))
    with s set by bisection so mean(w) = mean_deg.  Unordered pairs are drawn with
    endpoints i.i.d. proportional to w; self pairs dropped; duplicates merged; more
    pairs are drawn until the realised mean degree is within 2% of the target.
    Node ids are then relabelled by a seeded random permutation."""
    idx = np.arange(1, n + 1, dtype=np.float64)
    base = idx ** (-1.0 / (gamma - 1.0))
    lo, hi = 0.0, float(cap) / base[0] * 4.0 + mean_deg * n
    for _ in range(80):
        s = 0.5 * (lo + hi)
        if np.minimum(cap, s * base).mean() < mean_deg:
            lo = s
        else:
            hi = s
    w = np.minimum(cap, s * base)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    target_pairs = n * mean_deg / 2.0
    keys = np.empty(0, np.int64)
    draw = int(round(target_pairs))
    for _ in range(8):
        a = np.searchsorted(cdf, rng.random(draw), side="right")
        b = np.searchsorted(cdf, rng.random(draw), side="right")
        a = np.minimum(a, n - 1)
        b = np.minimum(b, n - 1)
        m = a != b
        a, b = a[m], b[m]
        lo_ = np.minimum(a, b).astype(np.int64)
        hi_ = np.maximum(a, b).astype(np.int64)
        keys = np.unique(np.concatenate([keys, lo_ * n + hi_]))
        if keys.size >= 0.98 * target_pairs:
            break
        draw = int((target_pairs - keys.size) * 1.3) + 1
    perm = rng.permutation(n).astype(np.int64)
    u = perm[keys // n]
    v = perm[keys % n]
    return u, v


def _tiny(seed_g, seed_x, n=2048, F=64):
    rng = _rng(seed_g)
    u, v = _erdos_renyi_pairs(rng, n, 4.0 / (n - 1))
    row, col = _sym_with_self(u, v, n)
    val = _gcn_values(row, col, n)
    X = _um11(_rng(seed_x), (n, F))
    return row, col, val, X, dict(n=n, F=F, p=4.0 / (n - 1), symmetric=True)


def _powerlaw(seed_g, seed_x, n=100_000, F=128, gamma=2.1, mean_deg=10.0, cap=5000):
    rng = _rng(seed_g)
    u, v = _chung_lu_pairs(rng, n, gamma, mean_deg, cap)
    row, col = _sym_with_self(u, v, n)
    val = _gcn_values(row, col, n)
    X = _normal(_rng(seed_x), (n, F))
    return row, col, val, X, dict(n=n, F=F, gamma=gamma, mean_deg=mean_deg, cap=cap, symmetric=True)


def _mesh(seed_g, seed_x, m=512, F=64):
    n = m * m
    ids = np.arange(n, dtype=np.int64)
    r, c = ids // m, ids % m
    parts = [ids * n + ids]
    for dr, dc in ((-1, 0), (1, 0), (0, -1), (0, 1)):
        ok = (r + dr >= 0) & (r + dr < m) & (c + dc >= 0) & (c + dc < m)
        parts.append(ids[ok] * n + (ids[ok] + dr * m + dc))
    row, col = _canon_from_keys(np.concatenate(parts), n)
    val = _u01_closed_top(_rng(seed_g), row.size)
    X = _um11(_rng(seed_x), (n, F))
    return row, col, val, X, dict(n=n, m=m, F=F, symmetric=False)


def _blocks(seed_g, seed_x, n_comm=12_800, size=16, F=256, p=0.8, inter=2):
    n = n_comm * size
    rng = _rng(seed_g)
    li, lj = np.triu_indices(size, k=1)
    keep = rng.random((n_comm, li.size)) < p
    base = (np.arange(n_comm, dtype=np.int64) * size)[:, None]
    u_in = (base + li[None, :])[keep]
    v_in = (base + lj[None, :])[keep]
    src = np.repeat(np.arange(n, dtype=np.int64), inter)
    comm = src // size
    draw = rng.integers(0, n - size, size=src.size, dtype=np.int64)
    dst = np.where(draw >= comm * size, draw + size, draw)  # skip own community
    u = np.concatenate([u_in, src])
    v = np.concatenate([v_in, dst])
    row, col = _sym_with_self(u, v, n)
    val = _gcn_values(row, col, n)
    X = _normal(_rng(seed_x), (n, F))
    return row, col, val, X, dict(n=n, n_comm=n_comm, size=size, F=F, p=p, inter=inter, symmetric=True)


def _large(seed_g, seed_x, n=2_000_000, F=128, gamma=2.0, mean_deg=25.0, cap=None):
    if cap is None:
        cap = int(math.floor(math.sqrt(n * mean_deg)))
    rng = _rng(seed_g)
    u, v = _chung_lu_pairs(rng, n, gamma, mean_deg, cap)
    row, col = _sym_with_self(u, v, n)
    raw = _u01_open(rng, row.size).astype(np.float64)
    rs = np.bincount(row, weights=raw, minlength=n)
    val = (raw / rs[row]).astype(np.float32)
    X = _normal(_rng(seed_x), (n, F))
    return row, col, val, X, dict(n=n, F=F, gamma=gamma, mean_deg=mean_deg, cap=cap, symmetric=False)


_BUILDERS = {1: _tiny, 2: _powerlaw, 3: _mesh, 4: _blocks, 5: _large}

# Scaled-down shapes of the same recipes, small enough for the oracle to
# finish in seconds but still spanning many tiles with ragged tails.
_SCALED = {
    1: dict(n=2048),
    2: dict(n=6007, cap=400),
    3: dict(m=77),
    4: dict(n_comm=301),
    5: dict(n=20_011),
}


@functools.lru_cache(maxsize=4)
def config(k: int) -> Graph:
    """Full-size workload k (1..5); seeds 1000+k (graph) and 2000+k (X)."""
    row, col, val, X, meta = _BUILDERS[k](1000 + k, 2000 + k)
    n = X.shape[0]
    return Graph(CONFIG_NAMES[k], n, n, row, col, val, X, meta)


@functools.lru_cache(maxsize=8)
def scaled(k: int) -> Graph:
    """Scaled-down workload k with the same recipe (and its own seeds)."""
    row, col, val, X, meta = _BUILDERS[k](1100 + k, 2100 + k, **_SCALED[k])
    n = X.shape[0]
    return Graph(CONFIG_NAMES[k] + "-scaled", n, n, row, col, val, X, meta)


def layer2_input(Y1: np.ndarray, seed: int = 3005) -> np.ndarray:
    """Second-layer input of the large workload: ReLU(Y1 @ W), W ~ N(0, 1/F)."""
    F = Y1.shape[1]
    W = (_rng(seed).standard_normal((F, F)) / math.sqrt(F)).astype(np.float32)
    return np.maximum(Y1 @ W, 0.0).astype(np.float32)


def layer2_weight(F: int, seed: int = 3005) -> np.ndarray:
    return (_rng(seed).standard_normal((F, F)) / math.sqrt(F)).astype(np.float32)


def random_coo(R: int, C: int, nnz: int, seed: int, empty_rows: float = 0.0,
               values: str = "normal"):
    """Random canonical COO with exactly min(nnz, R*C) distinct entries.

    ``empty_rows`` is the fraction of rows forced empty.  Values are never
    zero ("normal" draws N(0,1) and replaces exact zeros by 1)."""
    rng = _rng(seed)
    allowed = np.arange(R, dtype=np.int64)
    if empty_rows > 0 and R > 0:
        allowed = allowed[rng.random(R) >= empty_rows]
    if allowed.size == 0 or C == 0:
        z = np.zeros(0, np.int32)
        return z, z.copy(), np.zeros(0, np.float32)
    cap = allowed.size * C
    nnz = min(nnz, cap)
    keys = np.empty(0, np.int64)
    while keys.size < nnz:
        need = nnz - keys.size
        r = allowed[rng.integers(0, allowed.size, size=need * 2 + 8)]
        c = rng.integers(0, C, size=r.size)
        keys = np.unique(np.concatenate([keys, r * C + c]))
    if keys.size > nnz:
        keys = np.sort(rng.choice(keys, size=nnz, replace=False))
    row = (keys // C).astype(np.int32)
    col = (keys % C).astype(np.int32)
    if values == "normal":
        val = rng.standard_normal(row.size).astype(np.float32)
        val[val == 0] = 1.0
    else:
        val = _u01_open(rng, row.size)
    return row, col, val


def dense_rows_coo(R: int, C: int, dense_rows, seed: int, base_nnz: int = 0):
    """Canonical COO with the listed rows fully dense plus random background."""
    rng = _rng(seed)
    r0, c0, _ = random_coo(R, C, base_nnz, seed + 7)
    keys = [r0.astype(np.int64) * C + c0]
    for r in dense_rows:
        keys.append(np.int64(r) * C + np.arange(C, dtype=np.int64))
    keys = np.unique(np.concatenate(keys))
    row = (keys // C).astype(np.int32)
    col = (keys % C).astype(np.int32)
    val = _u01_open(rng, row.size)
    return row, col, val


def band_far_coo(n: int, band=(-2, 0, 3), seed: int = 0):
    """Canonical COO of an n x n matrix: (i, i+o) for every offset o in
    ``band`` that stays inside the matrix, plus (i, (i + n//2) mod n), a far
    diagonal that switches offset at row n - n//2.  Values uniform[-1,1),
    exact zeros replaced by 1/2."""
    rng = _rng(seed)
    i = np.arange(n, dtype=np.int64)
    keys = [i * n + (i + n // 2) % n]
    for o in band:
        ok = (i + o >= 0) & (i + o < n)
        keys.append(i[ok] * n + i[ok] + o)
    row, col = _canon_from_keys(np.concatenate(keys), n)
    val = _um11(rng, row.size)
    val[val == 0] = 0.5
    return row, col, val


def shuffled(row, col, val, seed: int):
    """The same triplets in a seeded random order (a non-canonical input)."""
    p = _rng(seed).permutation(row.size)
    return row[p].copy(), col[p].copy(), val[p].copy()


def features_x(n: int, F: int, seed: int, kind: str = "um11") -> np.ndarray:
    rng = _rng(seed)
    if kind == "normal":
        return _normal(rng, (n, F))
    if kind == "ones":
        return np.ones((n, F), np.float32)
    return _um11(rng, (n, F))


# ---------------------------------------------------------------- training set
# Matrices for training the format predictor.  The paper's recipe: square
# random 0/1 matrices, sizes 1,000..15,000 in steps of 200, "sparsity" 0.1% to
# 70%, read as density, here log-uniform and capped so that nnz <= 30M.  All
# stored values are 1 (the paper's 0/1 matrices).

TRAIN_SIZES = list(range(1000, 15001, 200))
TRAIN_NNZ_CAP = 30_000_000


def _bernoulli_rows(rng, n, d, chunk=512):
    rows, cols = [], []
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        m = rng.random((r1 - r0, n)) < d
        rr, cc = np.nonzero(m)
        rows.append((rr + r0).astype(np.int32))
        cols.append(cc.astype(np.int32))
    return np.concatenate(rows), np.concatenate(cols)


def training_matrix(i: int):
    """Training matrix i (0..299) of the random 0/1 recipe: (n, row, col, val, meta)."""
    rng = _rng(50_000 + i)
    n = TRAIN_SIZES[i % len(TRAIN_SIZES)]
    d = float(np.exp(rng.uniform(np.log(1e-3), np.log(0.7))))
    d = min(d, TRAIN_NNZ_CAP / float(n * n))
    if d > 0.02:
        row, col = _bernoulli_rows(rng, n, d)
    else:
        k = int(rng.binomial(n * n, d))
        keys = np.unique(rng.integers(0, n * n, size=k, dtype=np.int64))
        row, col = (keys // n).astype(np.int32), (keys % n).astype(np.int32)
    if row.size == 0:
        row, col = np.zeros(1, np.int32), np.zeros(1, np.int32)
    return n, row, col, np.ones(row.size, np.float32), dict(kind="random01", density=d)


LARGE_SIZE_RANGE = (15000, 60000)


def large_training_matrix(i: int):
    """Large training matrix i (0..99): random 0/1, n log-uniform in
    15,000..60,000 (GNN graph sizes, above the paper's 15,000), density
    log-uniform in 0.01%..10% (nnz capped at 30M).  Disjoint seeds from the
    evaluation matrices."""
    rng = _rng(80_000 + i)
    lo, hi = LARGE_SIZE_RANGE
    n = int(round(float(np.exp(rng.uniform(np.log(lo), np.log(hi))))))
    d = float(np.exp(rng.uniform(np.log(1e-4), np.log(0.1))))
    d = min(d, TRAIN_NNZ_CAP / float(n * n))
    if d > 0.02:
        row, col = _bernoulli_rows(rng, n, d)
    else:
        k = max(1, int(rng.binomial(n * n, d)))
        keys = np.unique(rng.integers(0, n * n, size=k, dtype=np.int64))
        row, col = (keys // n).astype(np.int32), (keys % n).astype(np.int32)
    return n, row, col, np.ones(row.size, np.float32), dict(kind="random01-large", density=d)


EVAL_SIZE_RANGE = (1000, 60000)


def evaluation_matrix(i: int):
    """Evaluation matrix i (0..99) of the held-out set with random float
    values: square, n log-uniform in 1,000..60,000 (beyond the training
    sizes, up to the size of the paper's largest dataset), density
    log-uniform in 0.01%..10% (nnz capped at 30M), stored values random
    floats in (0, 1] (the (0,1) recipe rounded to fp32).  Never used for
    training."""
    rng = _rng(70_000 + i)
    lo, hi = EVAL_SIZE_RANGE
    n = int(round(float(np.exp(rng.uniform(np.log(lo), np.log(hi))))))
    d = float(np.exp(rng.uniform(np.log(1e-4), np.log(0.1))))
    d = min(d, TRAIN_NNZ_CAP / float(n * n))
    if d > 0.02:
        row, col = _bernoulli_rows(rng, n, d)
    else:
        k = max(1, int(rng.binomial(n * n, d)))
        keys = np.unique(rng.integers(0, n * n, size=k, dtype=np.int64))
        row, col = (keys // n).astype(np.int32), (keys % n).astype(np.int32)
    return n, row, col, _u01_open(rng, row.size), dict(kind="random-float", density=d)


def structured_matrix(i: int):
    """Structured training matrix i: banded, community-block, power-law and
    grid patterns, values 1.  Matrices 0..119 have 10^4..2x10^5 rows,
    matrices 120..159 have 2x10^5..1.5x10^6 (the sizes of large GNN graphs;
    banded ones then keep at most 30 diagonals, power-law ones have expected
    degrees capped at 1..8 x sqrt(n deg) instead of sqrt(n deg))."""
    rng = _rng(60_000 + i)
    kind = ("banded", "blocks", "powerlaw", "grid")[i % 4]
    lo, hi = (1e4, 2e5) if i < 120 else (2e5, 1.5e6)
    n = int(np.exp(rng.uniform(np.log(lo), np.log(hi))))
    if kind == "banded":
        nd = int(rng.integers(1, 40 if i < 120 else 30))
        offs = np.unique(rng.integers(-n // 8, n // 8, size=nd))
        keys = []
        for o in offs:
            r = np.arange(max(0, -o), min(n, n - o), dtype=np.int64)
            keep = rng.random(r.size) < rng.uniform(0.6, 1.0)
            keys.append(r[keep] * n + r[keep] + o)
        row, col = _canon_from_keys(np.concatenate(keys), n)
    elif kind == "blocks":
        size = int(rng.choice([4, 8, 16, 32]))
        nc = max(1, n // size)
        n = nc * size
        p = rng.uniform(0.2, 1.0)
        li, lj = np.triu_indices(size, k=0)
        keep = rng.random((nc, li.size)) < p
        base = (np.arange(nc, dtype=np.int64) * size)[:, None]
        u = (base + li[None, :])[keep]
        v = (base + lj[None, :])[keep]
        inter = int(rng.integers(0, 6))
        src = np.repeat(np.arange(n, dtype=np.int64), inter)
        dst = rng.integers(0, n, size=src.size, dtype=np.int64)
        row, col = _sym_with_self(np.concatenate([u, src]), np.concatenate([v, dst]), n)
    elif kind == "powerlaw":
        gamma = rng.uniform(1.8, 3.0)
        deg = rng.uniform(3, 30)
        cap = np.sqrt(n * deg)
        if i >= 120:  # hub-heavy too: expected degrees capped at 1..8 x sqrt(n deg)
            cap *= rng.uniform(1.0, 8.0)
        u, v = _chung_lu_pairs(rng, n, gamma, deg, int(cap))
        row, col = _sym_with_self(u, v, n)
    else:
        m = int(np.sqrt(n))
        n = m * m
        ids = np.arange(n, dtype=np.int64)
        r, c = ids // m, ids % m
        parts = [ids * n + ids]
        for dr, dc in ((-1, 0), (1, 0), (0, -1), (0, 1), (-1, -1), (1, 1))[: int(rng.integers(2, 7))]:
            ok = (r + dr >= 0) & (r + dr < m) & (c + dc >= 0) & (c + dc < m)
            parts.append(ids[ok] * n + (ids[ok] + dr * m + dc))
        row, col = _canon_from_keys(np.concatenate(parts), n)
    return n, row, col, np.ones(row.size, np.float32), dict(kind=kind)
