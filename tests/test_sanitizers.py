"""CPU builds under AddressSanitizer and UndefinedBehaviorSanitizer:

* the library's host-only arithmetic (csrc/gs_model.cpp: the predictor's
  model parser and tree walk; csrc/gs_featmath.cpp: the Table 2 doubles),
  driven by tests/c/host_fuzz.cpp over the shipped and built-in models,
  every truncation of them and garbled variants, and edge-case aggregates;
* the oracle (oracle/oracle.c), running its pin tests in a child process
  with the sanitizer runtime preloaded.
"""
import os
import shutil
import subprocess
import sys

import pytest

from conftest import ROOT

CSRC = os.path.join(ROOT, "paper_2111_00352_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _asan_runtime():
    p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return p if p and os.path.isabs(p) and os.path.exists(p) else None


pytestmark = pytest.mark.skipif(shutil.which("g++") is None or _asan_runtime() is None,
                                reason="g++ with the sanitizer runtimes is needed")


def test_host_arithmetic_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_fuzz")
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-g", *SAN, "-Wall", "-Wextra", "-Werror", "-o", exe,
                           os.path.join(ROOT, "tests", "c", "host_fuzz.cpp"),
                           os.path.join(CSRC, "gs_model.cpp"), os.path.join(CSRC, "gs_featmath.cpp")])
    model = os.path.join(ROOT, "paper_2111_00352_amd", "selector", "model.gsm")
    r = subprocess.run([exe, model], capture_output=True, text=True, timeout=600,
                       env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"})
    assert r.returncode == 0, r.stderr[-4000:]
    assert "host_fuzz ok" in r.stdout
    parsed, refused = (int(w) for w in r.stdout.split(":")[1].replace("parsed,", "").replace("refused", "").split())
    assert parsed > 0 and refused > 0


def test_oracle_under_sanitizers():
    env = {**os.environ, "ORACLE_SANITIZE": "1", "LD_PRELOAD": _asan_runtime(),
           "ASAN_OPTIONS": "detect_leaks=0", "OMP_NUM_THREADS": "4"}
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_gcn.py")],
                       capture_output=True, text=True, timeout=900, cwd=ROOT, env=env)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout
