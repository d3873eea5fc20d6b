"""Profile the training matrices on the GPU: features + per-format SpMM time.

Usage: python -m paper_2111_00352_amd.selector.collect OUT.csv [--random N] [--structured M] [--large L] [--eval E]

Each (matrix, F) row holds the Table 2 features (Sec. 4.4), the 16x16 block
count, F, and the median time of every storage format measured by the
library's exhaustive selector (inf where a format exceeds the memory cap).
Labelling is Eq. 1 with w = 1 (time only), done by ``train``.
"""
import argparse
import csv
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import graphgen  # noqa: E402
import paper_2111_00352_amd as gs  # noqa: E402

FMT = ["coo", "csr", "ell", "dia", "bsr"]
HEADER = (["set", "index", "kind", "n", "nnz", "F"] + gs.FEATURE_NAMES + ["n_blocks16"]
          + [f"t_{f}" for f in FMT])


def profile(n, row, col, val, F, key, reps):
    dev = "cuda"
    r, c, v = (torch.from_numpy(a).to(dev) for a in (row, col, val))
    X = torch.randn(n, F, device=dev)
    feats = gs.extract_features(r, c, v, (n, n))
    ctx = gs.SelectContext("profile", profile_reps=reps, formats=FMT)
    ctx.run(key, r, c, v, (n, n), X)
    st = ctx.stats()
    ctx.close()
    times = [st["scores"][f] if st["scores"][f] > 0 else math.inf for f in FMT]
    return feats, times


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("out")
    ap.add_argument("--random", type=int, default=300)
    ap.add_argument("--structured", type=int, default=160)
    ap.add_argument("--large", type=int, default=100,
                    help="random 0/1 matrices of 15,000..60,000 rows (graphgen.large_training_matrix)")
    ap.add_argument("--eval", type=int, default=0,
                    help="held-out matrices with random float values (graphgen.evaluation_matrix)")
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--start", type=int, default=0, help="first job (to split a collection)")
    ap.add_argument("--count", type=int, default=None, help="number of jobs from --start")
    a = ap.parse_args()
    torch.cuda.set_device(0)
    jobs = [("random", i, (64, 128)) for i in range(a.random)]
    jobs += [("structured", i, (64, 128, 256)) for i in range(a.structured)]
    jobs += [("large", i, (64, 128)) for i in range(a.large)]
    jobs += [("eval", i, (64, 128)) for i in range(a.eval)]
    jobs = jobs[a.start:None if a.count is None else a.start + a.count]
    t0 = time.time()
    with open(a.out, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(HEADER)
        for k, (kind, i, Fs) in enumerate(jobs):
            gen = {"random": graphgen.training_matrix, "structured": graphgen.structured_matrix,
                   "large": graphgen.large_training_matrix, "eval": graphgen.evaluation_matrix}[kind]
            n, row, col, val, meta = gen(i)
            for F in Fs:
                feats, times = profile(n, row, col, val, F, k, a.reps)
                w.writerow([kind, i, meta["kind"], n, row.size, F] + feats["f"] + [feats["n_blocks16"]]
                           + [f"{t:.9g}" for t in times])
            fh.flush()
            torch.cuda.empty_cache()
            print(f"[{k + 1}/{len(jobs)}] {kind} {i} n={n} nnz={row.size} "
                  f"best={FMT[int(np.argmin(times))]} t={time.time() - t0:.0f}s", flush=True)


if __name__ == "__main__":
    main()
