#!/usr/bin/env python3
"""SpMM benchmark: GNN aggregation Y = A.X with per-layer format selection.

One step = one GNN layer's aggregation through the selector
(gs_select_and_run) on one batch of features, with the adjacency's features,
prediction and format conversion already cached from the warm-up (the paper
decides the format once per layer across epochs, Sec. 5.2); those first-call
costs are measured and reported separately.  Steps rotate over several
(X, Y) batches so that consecutive steps do not find their operands in the
256 MiB last-level cache.

Headline workload: the power-law graph (n = 100,000, Chung-Lu exponent 2.1,
mean degree 10, GCN-normalised fp32, X 100,000 x 128 fp32).  Also reported:
every format's SpMM time on the same workload, the selector's speedup over
fixed CSR, the roofline fraction of the dominant kernel, and the CPU oracle's
throughput on this machine's cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s

WORKLOADS = {
    1: "tiny ER GCN n=2048 F=64",
    2: "power-law Chung-Lu n=100000 gamma=2.1 deg=10 GCN F=128",
    3: "mesh 512x512 5-point n=262144 F=64",
    4: "block-community n=204800 (16-node blocks p=0.8, 2 inter/node) GCN F=256",
    5: "large Chung-Lu n=2000000 gamma=2.0 deg=25 row-stochastic F=128 (layer 1)",
}


WORKLOAD_KEYS = {1: "tiny", 2: "powerlaw", 3: "mesh", 4: "blocks", 5: "large"}


def b_alg(R, C, Z, F):
    """Algorithmic bytes of one SpMM: CSR-equivalent A, X read once, Y written once."""
    return 4 * (R + 1) + 8 * Z + 4 * C * F + 4 * R * F


def time_launches(fn, stream, reps, inputs):
    """Per-launch durations (s) of fn(i) measured with HIP events on `stream`."""
    import torch

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for i in range(reps):
        ev[i][0].record(stream)
        fn(inputs[i % len(inputs)])
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    return np.array([a.elapsed_time(b) * 1e-3 for a, b in ev])


def cpu_baseline(g, F, budget_s=10.0):
    """The oracle's SpMM on this host: all threads for about budget_s, then
    one thread for a quarter of that (the results are identical)."""
    import oracle

    rp = oracle.csr(g.R, g.row)
    X = g.X[:, :F]

    def rate(budget):
        t0 = time.perf_counter()
        reps = 0
        while True:
            oracle.spmm(g.R, rp, g.col, g.val, X)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget:
                return 2.0 * g.nnz * F * reps / el / 1e9, reps, el

    threads = oracle.num_threads()
    v, reps, el = rate(budget_s)
    oracle.set_threads(1)
    v1, reps1, el1 = rate(budget_s / 4)
    oracle.set_threads(threads)
    return {
        "value": round(v, 3),
        "unit": "GFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"full {g.R}-row SpMM (fp64 accumulation, plus |A||X|) repeated {reps}x in {el:.1f}s "
                  f"on {threads} threads; single thread: {reps1}x in {el1:.1f}s",
        "single_thread_value": round(v1, 3),
    }


def gcn_e2e(g, row, col, val, X, args, hidden=128, out_dim=64):
    """Two-layer GCN trained for 10 epochs (Sec. 5.2) with the selector and with
    fixed CSR / COO, each from a fresh context so every first-call cost is
    inside its total."""
    import torch

    import graphgen
    from paper_2111_00352_amd import gcn

    torch.backends.cuda.matmul.allow_tf32 = False
    dev = X.device
    F = X.shape[1]
    W1 = torch.from_numpy(graphgen.features_x(F, hidden, 4100, "normal")).to(dev) / F ** 0.5
    W2 = torch.from_numpy(graphgen.features_x(hidden, out_dim, 4200, "normal")).to(dev) / hidden ** 0.5
    T = torch.from_numpy(graphgen.features_x(g.R, out_dim, 4300, "normal")).to(dev)
    res = gcn.end_to_end(row, col, val, (g.R, g.C), X, T, W1, W2, epochs=args.gcn_epochs, lr=0.1,
                         symmetric=bool(g.meta.get("symmetric", False)))
    r = {"epochs": args.gcn_epochs, "hidden": hidden, "out": out_dim}
    for k, v in res.items():
        if isinstance(v, dict):
            r[k] = {"total_ms": round(v["total_s"] * 1e3, 3), "first_epoch_ms": round(v["first_epoch_s"] * 1e3, 3),
                    "steady_epoch_ms": round(v["steady_epoch_s"] * 1e3, 3), "formats": v["formats"],
                    "final_loss": round(v["final_loss"], 6)}
        else:
            r[k] = round(v, 3)
    return r


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, help="workload 1..5 (default: power-law)")
    ap.add_argument("--batches", type=int, default=4, help="rotating (X, Y) batches")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--format-reps", type=int, default=50)
    ap.add_argument("--no-gcn", action="store_true", help="skip the two-layer GCN end-to-end run")
    ap.add_argument("--gcn-epochs", type=int, default=10)
    ap.add_argument("--profile-run", action="store_true",
                    help="only run the timed steps plus a 256 MiB calibration copy (for rocprofv3)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: runs on one GPU only (there is no multi-GPU path); use --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import graphgen
    import paper_2111_00352_amd as gs

    assert torch.cuda.is_available(), "bench needs a GPU"
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream()

    t_gen = time.perf_counter()
    g = graphgen.config(args.config)
    t_gen = time.perf_counter() - t_gen
    R, C, Z, F = g.R, g.C, g.nnz, g.F
    row = torch.from_numpy(g.row).to(dev)
    col = torch.from_numpy(g.col).to(dev)
    val = torch.from_numpy(g.val).to(dev)
    Xs, Ys = [], []
    rng = np.random.default_rng(7)
    for b in range(args.batches):
        X = torch.from_numpy(g.X if b == 0 else rng.permutation(g.X, axis=0)).to(dev)
        Xs.append(X)
        Ys.append(torch.empty((R, F), dtype=torch.float32, device=dev))
    torch.cuda.synchronize()

    flops = 2.0 * Z * F
    balg = b_alg(R, C, Z, F)

    # ---- one-time library start-up (code objects loaded on first launch),
    # paid once per process, not per matrix: taken on a small identity matrix
    t0 = time.perf_counter()
    n0 = 256
    i0 = torch.arange(n0, dtype=torch.int32, device=dev)
    warm = gs.SelectContext("model")
    for fmt_probe in ("csr", "coo", "ell", "dia", "bsr", "csc"):
        gs.build_format(i0, i0, torch.ones(n0, device=dev), (n0, n0), fmt_probe).spmm(
            torch.ones((n0, F), device=dev))
    warm.run(0, i0, i0, torch.ones(n0, device=dev), (n0, n0), torch.ones((n0, F), device=dev))
    torch.cuda.synchronize()
    warm.close()
    library_init_s = time.perf_counter() - t0

    # ---- selector: first call (features + prediction + conversion), then steady state
    ctx = gs.SelectContext("model")
    t0 = time.perf_counter()
    _, chosen = ctx.run(1, row, col, val, (R, C), Xs[0], out=Ys[0])
    torch.cuda.synchronize()
    first_call_s = time.perf_counter() - t0
    st = ctx.stats()

    def step(i):
        return ctx.run(1, row, col, val, (R, C), Xs[i % args.batches], out=Ys[i % args.batches])

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    ms_per_step = el / args.steps * 1e3
    value = flops / (el / args.steps) / 1e9
    if args.profile_run:
        # plain elementwise copy of known size: calibrates the byte counters
        src = torch.ones(64 * 2**20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print(f"profile run: {args.steps} steps of spmm_{chosen}, {ms_per_step * 1e3:.2f} us/step", flush=True)
        return

    # ---- per-launch duration of the chosen format's SpMM (HIP events on its stream)
    mats = {}
    fmt_rows = {}
    for fmt in ("csr", "coo", "ell", "dia", "bsr", "csc"):
        try:
            t0 = time.perf_counter()
            m = gs.build_format(row, col, val, (R, C), fmt)
            torch.cuda.synchronize()
            t_build = time.perf_counter() - t0
        except gs.GnnSpmmError as e:
            fmt_rows[fmt] = {"feasible": False, "bytes_required": getattr(e, "bytes_required", None)}
            continue
        mats[fmt] = m
        pairs = list(zip(Xs, Ys))
        for i in range(3):
            m.spmm(*pairs[i % len(pairs)][:1], out=pairs[i % len(pairs)][1])
        d = time_launches(lambda p: m.spmm(p[0], out=p[1]), stream, args.format_reps, pairs)
        t = float(np.median(d))
        fmt_rows[fmt] = {
            "feasible": True, "median_us": round(t * 1e6, 2), "min_us": round(float(d.min()) * 1e6, 2),
            "p90_us": round(float(np.percentile(d, 90)) * 1e6, 2),
            "gflops": round(flops / t / 1e9, 1), "roofline_frac": round(balg / t / 1e9 / HBM_PEAK_GBS, 4),
            "format_bytes": m.device_bytes, "build_s": round(t_build, 4),
        }
    d_sel = time_launches(lambda p: ctx.run(1, row, col, val, (R, C), p[0], out=p[1]), stream,
                          args.format_reps, list(zip(Xs, Ys)))
    t_sel = float(np.median(d_sel))
    feasible = {k: v for k, v in fmt_rows.items() if v.get("feasible")}
    best = min(feasible, key=lambda k: feasible[k]["median_us"])
    t_csr = feasible["csr"]["median_us"]
    achieved = balg / t_sel / 1e9
    # amortised over 10 epochs of one layer (Sec. 5.2): the selector pays its
    # first call (features, prediction, conversion, one SpMM) once; fixed CSR
    # pays its build once
    epochs = 10
    e2e_sel = first_call_s + (epochs - 1) * t_sel
    e2e_csr = feasible["csr"]["build_s"] + epochs * feasible["csr"]["median_us"] * 1e-6

    traffic = None
    tpath = os.path.join(ROOT, "profiles", f"traffic_{WORKLOAD_KEYS[args.config]}_{chosen}.json")
    if os.path.exists(tpath):
        from paper_2111_00352_amd.profsum import source_hash

        with open(tpath) as f:
            tj = json.load(f)
        if tj.get("source_hash") == source_hash():
            traffic = round(tj["bytes"] / 1e6, 2)

    out = {
        "metric": "SpMM GFLOP/s (2*nnz*F) + % HBM roofline per format; best-vs-CSR speedup",
        "value": round(value, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.config], "n": R, "nnz": Z, "F": F,
                   "batches": args.batches},
        "roofline": {
            "bound": "hbm",
            "kernel": f"spmm_{chosen} (all launches of one SpMM)",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            # measured bytes over the same launch time: the rate the memory
            # system actually sustains for this kernel
            "traffic_rate_gbs": None if traffic is None else round(traffic * 1e6 / t_sel / 1e9, 1),
            "traffic_unit": "MB per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "bytes_per_launch": balg,
            "launch_us": round(t_sel * 1e6, 2),
        },
        "selector": {
            "mode": "model",
            "chosen": chosen,
            "best_measured": best,
            # steady-state kernel speedup of the chosen format over fixed CSR,
            # and of the best measured format (the exhaustive-search reference)
            "speedup_vs_csr": round(t_csr / feasible[chosen]["median_us"], 3),
            "best_vs_csr": round(t_csr / feasible[best]["median_us"], 3),
            "fraction_of_best": round(feasible[best]["median_us"] / feasible[chosen]["median_us"], 3),
            "speedup_vs_coo": round(feasible["coo"]["median_us"] / feasible[chosen]["median_us"], 3),
            "amortised_speedup_vs_csr_10_epochs": round(e2e_csr / e2e_sel, 3),
            "selector_step_us": round(t_sel * 1e6, 2),
            "host_overhead_us": round(t_sel * 1e6 - feasible[chosen]["median_us"], 2),
            "first_call_s": round(first_call_s, 4),
            "library_init_s": round(library_init_s, 4),
            "t_features_s": round(st["t_features"], 4),
            "t_predict_us": round(st["t_predict"] * 1e6, 2),
            "t_convert_s": round(st["t_convert"], 4),
        },
        "formats": fmt_rows,
        "gen_s": round(t_gen, 2),
        "device": torch.cuda.get_device_name(0),
        "arch": getattr(torch.cuda.get_device_properties(0), "gcnArchName", None),
        "compute_units": torch.cuda.get_device_properties(0).multi_processor_count,
        "hip": torch.version.hip,
    }
    if not args.no_gcn:
        out["gcn_e2e"] = gcn_e2e(g, row, col, val, Xs[0], args)
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(g, F, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
