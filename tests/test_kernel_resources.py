"""Every HIP kernel fits its registers: the compiler's resource report for
gfx950 shows no scratch (register spill) in any kernel instantiation.

Compiles the library's device code once (about a minute, no GPU needed)."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_29119_amd", "csrc")


def test_no_kernel_spills(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    from paper_2609_29119_amd.build import HIP_FLAGS
    cmd = [hipcc, *HIP_FLAGS, "--cuda-device-only", "-c", os.path.join(CSRC, "nsgcqt.hip"),
           "-o", str(tmp_path / "dev.o"), "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stderr[-2000:]
    names = re.findall(r"Function Name: (\S+)", r.stderr)
    scratch = [int(v) for v in re.findall(r"ScratchSize \[bytes/lane\]: (\d+)", r.stderr)]
    assert names and len(names) == len(scratch)
    spilled = [(n, s) for n, s in zip(names, scratch) if s]
    assert not spilled, spilled
