"""The C ABI from a C99 program: the header compiles as C and the library
links and answers host-only calls (no GPU needed)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2609_29119_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_c_client_of_host_only_plans(tmp_path):
    if not os.path.exists(os.path.join(LIB_DIR, "libnsgcqt.so")):
        pytest.fail("libnsgcqt.so is not built; run python -m paper_2609_29119_amd.build")
    exe = tmp_path / "abi_host"
    cmd = ["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c", "abi_host.c"), "-o", str(exe),
           "-L", LIB_DIR, "-lnsgcqt", "-Wl,-rpath," + LIB_DIR, "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "ok"
