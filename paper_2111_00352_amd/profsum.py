"""Summarise rocprofv3 result databases (rocpd SQLite) into short text.

Usage:
  python -m paper_2111_00352_amd.profsum --trace TRACE.db [--fetch FETCH.db --write WRITE.db]
         [--kernel SUBSTR] [--calib-bytes N] [--traffic-json OUT.json] [--cmd "..."]

--trace: a ``--kernel-trace --stats`` run; per-kernel dispatch count and
average / median / min duration.
--fetch / --write: ``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE`` runs; the
counters (KiB per dispatch) are averaged per kernel and scaled by what the
same counter reads for the calibration kernel, a plain elementwise copy
(``neg``) of --calib-bytes read and written.  With --traffic-json the scaled
bytes per dispatch of the kernels matching --kernel are written out together
with a hash of the HIP sources they were measured on.
"""
from __future__ import annotations

import argparse
import collections
import glob
import hashlib
import json
import os
import sqlite3

HERE = os.path.dirname(os.path.abspath(__file__))


def source_hash() -> str:
    """Hash of the device code: the HIP sources and the headers they include
    (host-only .cpp files -- ABI glue, selector -- do not change a kernel)."""
    h = hashlib.sha256()
    files = glob.glob(os.path.join(HERE, "csrc", "*.hip")) + glob.glob(os.path.join(HERE, "csrc", "*.h"))
    for p in sorted(files):
        with open(p, "rb") as f:
            h.update(os.path.basename(p).encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def _rows(db, view):
    cur = db.cursor()
    cols = [r[1] for r in cur.execute(f"pragma table_info({view})")]
    return [dict(zip(cols, r)) for r in cur.execute(f"select * from {view}")]


def kernel_times(path):
    db = sqlite3.connect(path)
    k = collections.defaultdict(list)
    for d in _rows(db, "kernels"):
        name = d.get("kernel_name") or d.get("name")
        k[name].append((d["end"] - d["start"]) / 1e3)
    return k


def counters(path):
    db = sqlite3.connect(path)
    agg = collections.defaultdict(list)
    for d in _rows(db, "counters_collection"):
        agg[(d.get("kernel_name"), d.get("counter_name"))].append(float(d.get("value")))
    return agg


def short(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "")
    return name.split("(")[0] if "(" in name else name


def picked(name: str, kernels) -> bool:
    """True when the kernel's name (template arguments included, without the
    return type and namespace) is one of `kernels`."""
    return short(str(name)).split("gs::")[-1] in kernels


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--kernel", default="k_csr_rows<4, 32, true>;k_csr_combine<4, 32>",
                    help="kernel names (with template arguments) of one SpMM, separated by ;")
    ap.add_argument("--calib-bytes", type=float, default=256 * 2**20)
    ap.add_argument("--traffic-json")
    ap.add_argument("--counters", nargs="*", default=[],
                    help="further --pmc runs: every counter averaged per dispatch of the --kernel kernels")
    ap.add_argument("--top", type=int, default=25, help="kernels listed from the trace (by total time)")
    ap.add_argument("--cmd", default="")
    a = ap.parse_args()
    kernels = [k.strip() for k in a.kernel.split(";")]
    if a.cmd:
        print(f"command: {a.cmd}")
    if a.trace:
        kt = kernel_times(a.trace)
        print(f"{'dispatches':>10} {'avg_us':>10} {'median_us':>10} {'min_us':>10}  kernel")
        for name, ds in sorted(kt.items(), key=lambda kv: -sum(kv[1]))[:a.top]:
            ds = sorted(ds)
            print(f"{len(ds):10d} {sum(ds) / len(ds):10.2f} {ds[len(ds) // 2]:10.2f} {ds[0]:10.2f}  {short(name)}")
    out = {}
    for label, path, cname in (("fetch", a.fetch, "FETCH_SIZE"), ("write", a.write, "WRITE_SIZE")):
        if not path:
            continue
        c = counters(path)
        calib = [sum(v) / len(v) for (kn, cn), v in c.items() if cn == cname and "neg" in str(kn)]
        factor = (a.calib_bytes / (max(calib) * 1024.0)) if calib else None
        print(f"\n{cname} (KiB per dispatch, averaged); calibration copy reads {calib and max(calib):.0f} KiB "
              f"for {a.calib_bytes / 1024:.0f} KiB moved -> factor {factor if factor else float('nan'):.4f}")
        for (kn, cn), v in sorted(c.items(), key=lambda kv: -sum(kv[1])):
            if cn != cname:
                continue
            avg = sum(v) / len(v)
            print(f"  {len(v):5d}x {avg:14.1f} KiB  {short(str(kn))}")
            if picked(kn, kernels) and factor:
                out[label] = out.get(label, 0.0) + avg * 1024.0 * factor
        if factor:
            out[f"{label}_factor"] = factor
    for path in a.counters:
        c = counters(path)
        print(f"\ncounters of *{a.kernel}* kernels (average per dispatch): {os.path.basename(os.path.dirname(path))}")
        per = collections.defaultdict(dict)
        for (kn, cn), v in sorted(c.items()):
            if picked(kn, kernels):
                per[short(str(kn))][cn] = sum(v) / len(v)
        for kn, cs in per.items():
            line = "  ".join(f"{cn}={val:.4g}" for cn, val in sorted(cs.items()))
            hit, miss = cs.get("TCC_HIT_sum"), cs.get("TCC_MISS_sum")
            if hit is not None and miss is not None and hit + miss > 0:
                line += f"  L2 hit rate={hit / (hit + miss):.3f}"
            print(f"  {kn}: {line}")
    if a.traffic_json and "fetch" in out and "write" in out:
        out["bytes"] = out["fetch"] + out["write"]
        out["kernel"] = a.kernel
        out["source_hash"] = source_hash()
        out["command"] = a.cmd
        with open(a.traffic_json, "w") as f:
            json.dump(out, f, indent=1)
        print(f"\ntraffic per dispatch of *{a.kernel}*: fetch {out['fetch'] / 1e6:.2f} MB + "
              f"write {out['write'] / 1e6:.2f} MB = {out['bytes'] / 1e6:.2f} MB")


if __name__ == "__main__":
    main()
