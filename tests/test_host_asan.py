"""The library's host code (argument checks, plan building, size queries) under
AddressSanitizer and UndefinedBehaviorSanitizer: the library is built with
host-side instrumentation only and driven by a C++ program on the CPU (no GPU
call is made).  Any memory error or undefined behaviour aborts the driver with
the sanitizer's report."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_07008_amd", "csrc")
from paper_2609_07008_amd.build import SOURCES   # every source of the library


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    pytest.skip("hipcc not found")


def test_host_code_under_asan(tmp_path):
    cc = _hipcc()
    common = ["-O1", "-g", "-std=c++17", "-I" + os.path.join(ROOT, "include"),
              "-Wno-unused-command-line-argument",
              "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=undefined",
              "-Xarch_host", "-fno-omit-frame-pointer"]
    lib = tmp_path / "libmla_asan.so"
    subprocess.run([cc, *common, "-fPIC", "-shared", "--offload-arch=gfx950",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-o", str(lib),
                    *[os.path.join(CSRC, s) for s in SOURCES]], check=True, capture_output=True)
    drv = tmp_path / "driver"
    subprocess.run([cc, *common, "-o", str(drv), os.path.join(ROOT, "tests", "host", "asan_driver.cpp"),
                    "-L" + str(tmp_path), "-lmla_asan", "-Wl,-rpath," + str(tmp_path)],
                   check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(drv)], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "random tables:" in r.stdout
