"""A property of the generated device code that the direct global->LDS loads
rely on (CPU only: hipcc cross-compiles gfx950).  Each such load sets m0 (its
LDS destination) inside its own asm statement; m0 is a register the compiler
reserves and does not preserve across asm, so this is only sound while the
compiler keeps no value of its own in m0 in those kernels.  The test compiles
each source that issues these loads to gfx950 assembly and checks that m0
appears only inside the asm statements."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_07008_amd", "csrc")


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    pytest.skip("hipcc not found")


def _sources_with_direct_loads():
    return sorted(f for f in os.listdir(CSRC)
                  if f.endswith(".hip") and "global_load_lds_dwordx4" in open(os.path.join(CSRC, f)).read())


def test_direct_load_sources_found():
    assert {"attend.hip", "wb.hip"} <= set(_sources_with_direct_loads())


@pytest.mark.parametrize("src", _sources_with_direct_loads())
def test_compiler_keeps_nothing_in_m0(src, tmp_path):
    from paper_2609_07008_amd.build import HIPCC_FLAGS
    out = tmp_path / "k.s"
    subprocess.run([_hipcc(), *HIPCC_FLAGS, "-Wno-inline-asm", "-I", CSRC, "--cuda-device-only", "-S",
                    os.path.join(CSRC, src), "-o", str(out)], check=True, capture_output=True)
    in_asm, outside = False, []
    for line in open(out):
        if ";;#ASMSTART" in line:
            in_asm = True
        elif ";;#ASMEND" in line:
            in_asm = False
        elif not in_asm and re.search(r"\bm0\b", line.split(";")[0]):
            outside.append(line.strip())
    assert not outside, outside[:10]
