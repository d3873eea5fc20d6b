"""The C ABI from plain C: tests/c/abi_check.c is compiled with gcc -std=c11
against include/gnnspmm.h, linked with the built library and run (host-side
checks only, no GPU)."""
import os
import subprocess

import paper_2111_00352_amd as gs
from conftest import ROOT


def test_c_caller_compiles_links_and_passes(tmp_path):
    if not os.path.exists(gs.library_path()):
        from paper_2111_00352_amd import build
        build.build()
    lib_dir = os.path.dirname(gs.library_path())
    exe = tmp_path / "abi_check"
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "abi_check.c"), "-o", str(exe),
                    "-L", lib_dir, "-lgnnspmm", f"-Wl,-rpath,{lib_dir}"], check=True)
    from paper_2111_00352_amd.selector import MODEL_PATH
    r = subprocess.run([str(exe), MODEL_PATH], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all checks passed" in r.stdout
