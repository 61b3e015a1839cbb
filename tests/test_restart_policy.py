"""The attention kernel's restart policy on the CPU (restart.h, compiled as host
code): a NaN weight sum never votes, +inf and sums >= 2^64 do, raises are
log2 of the sum or 128 after an overflow, and every work item makes at most
kMaxAttempts passes -- the property that keeps a non-finite input from holding
a workgroup in the tile loop forever."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    pytest.skip("hipcc not found")


def test_restart_policy(tmp_path):
    exe = tmp_path / "restart_policy"
    subprocess.run([_hipcc(), "-x", "hip", "-O1", "-std=c++17", "--offload-arch=gfx950",
                    "-I" + os.path.join(ROOT, "paper_2609_07008_amd", "csrc"), "-I" + os.path.join(ROOT, "include"),
                    "-Wno-unused-command-line-argument", "-o", str(exe),
                    os.path.join(ROOT, "tests", "host", "restart_policy.cpp")], check=True, capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "restart policy: 0 failure(s)" in r.stdout
