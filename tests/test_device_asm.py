"""Properties of the generated gfx950 device code (CPU only: hipcc cross-compiles
every library source to assembly once for the module).

* The direct global->LDS loads set m0 (their LDS destination) inside their own
  asm statements.  m0 is a register the compiler reserves and does not preserve
  across asm, so this is only sound while the compiler keeps no value of its
  own in m0 in the sources that issue them: m0 appears only inside the asm.
* No packed fp32 arithmetic (v_pk_add_f32, v_pk_mul_f32, v_pk_fma_f32): every
  source is built with the packed-fp32 feature turned off.
* No write through the scalar data cache: no scalar memory stores or atomics,
  and no write-back or discard of that cache; all stores are vector stores."""
import os
import re
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_07008_amd", "csrc")


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    pytest.skip("hipcc not found")


@pytest.fixture(scope="module")
def device_asm(tmp_path_factory):
    """source name -> list of (instruction text, inside an asm statement)"""
    from paper_2609_07008_amd.build import HIPCC_FLAGS, SOURCES
    cc = _hipcc()
    d = tmp_path_factory.mktemp("asm")

    def compile_one(src):
        out = d / (src + ".s")
        subprocess.run([cc, *HIPCC_FLAGS, "-Wno-inline-asm", "-I", CSRC, "--cuda-device-only", "-S",
                        os.path.join(CSRC, src), "-o", str(out)], check=True, capture_output=True)
        lines, in_asm = [], False
        for line in open(out):
            if ";;#ASMSTART" in line:
                in_asm = True
            elif ";;#ASMEND" in line:
                in_asm = False
            else:
                code = line.split(";")[0].strip()
                if code and not code.startswith("."):
                    lines.append((code, in_asm))
        return src, lines

    with ThreadPoolExecutor(max(1, min(len(SOURCES), os.cpu_count() or 1))) as ex:
        return dict(ex.map(compile_one, SOURCES))


def _direct_load_sources():
    return sorted(f for f in os.listdir(CSRC)
                  if f.endswith(".hip") and "global_load_lds_dwordx4" in open(os.path.join(CSRC, f)).read())


def test_direct_load_sources_found():
    assert {"attend.hip", "wb.hip"} <= set(_direct_load_sources())


def test_compiler_keeps_nothing_in_m0(device_asm):
    for src in _direct_load_sources():
        outside = [c for c, a in device_asm[src] if not a and re.search(r"\bm0\b", c)]
        assert not outside, (src, outside[:10])


def test_no_packed_fp32_arithmetic(device_asm):
    bad = [(s, c) for s, lines in device_asm.items() for c, _ in lines
           if re.match(r"v_pk_(add|mul|fma)_f32\b", c)]
    assert not bad, bad[:10]


def test_no_scalar_cache_writes(device_asm):
    bad = [(s, c) for s, lines in device_asm.items() for c, _ in lines
           if re.match(r"s_(store|buffer_store|scratch_store|atomic|buffer_atomic|dcache_wb|dcache_discard)", c)]
    assert not bad, bad[:10]
    # the library does store (so the pattern above sees real code): vector stores exist
    assert any(c.startswith("global_store") for lines in device_asm.values() for c, _ in lines)
