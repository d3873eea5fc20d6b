"""Host-side parts of bench.py (no GPU): the algorithmic byte count, the
one-GPU guard and the lookup of profiled traffic."""
import json
import os
import subprocess
import sys

from conftest import ROOT

sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2111_00352_amd.profsum import source_hash  # noqa: E402


def test_algorithmic_bytes():
    # CSR-equivalent A (row pointers, column indices, values), X read once, Y written once
    R, C, Z, F = 5, 7, 11, 3
    assert bench.b_alg(R, C, Z, F) == 4 * 6 + 8 * 11 + 4 * 7 * 3 + 4 * 5 * 3
    assert bench.b_alg(2_000_000, 2_000_000, 52_268_964, 128) == 2_474_151_716


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_profiled_traffic_needs_the_current_sources(tmp_path):
    os.makedirs(tmp_path / "profiles")
    assert bench.profiled_traffic("large", "csr", root=str(tmp_path)) is None  # no file
    path = tmp_path / "profiles" / "traffic_large_csr.json"
    path.write_text(json.dumps({"bytes": 22561840000.0, "source_hash": source_hash()}))
    assert bench.profiled_traffic("large", "csr", root=str(tmp_path)) == 22561.84
    path.write_text(json.dumps({"bytes": 22561840000.0, "source_hash": "0" * 16}))
    assert bench.profiled_traffic("large", "csr", root=str(tmp_path)) is None  # other sources


def test_committed_traffic_files_name_their_kernels_and_command():
    prof = os.path.join(ROOT, "profiles")
    files = [f for f in os.listdir(prof) if f.startswith("traffic_") and f.endswith(".json")]
    assert files
    for f in files:
        tj = json.load(open(os.path.join(prof, f)))
        assert tj["bytes"] > 0 and tj["kernel"] and "rocprofv3" in tj["command"], f
        assert abs(tj["fetch"] + tj["write"] - tj["bytes"]) < 1.0, f
