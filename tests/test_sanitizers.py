"""AddressSanitizer / UndefinedBehaviorSanitizer builds, run on the CPU:

* the oracle (gcc) over seeded random small layers, sampled points checked
  against whole tensors (tests/sanitize/oracle_checks.c);
* libdc's host code -- validation, tile geometry, halo bands, plans, sample
  groups, launch configuration -- compiled host-only and linked against a
  stub HIP runtime that checks every launch's configuration, over a few
  thousand seeded random problems (tests/sanitize/host_checks.c).
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_1903_06681_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/lib/llvm/bin/clang"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, (cmd[0], r.stdout[-3000:], r.stderr[-3000:])
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc missing")
def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_checks")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", *SAN_FLAGS, "-o", exe,
          os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(SAN, "oracle_checks.c")])
    r = _run([exe], env=ENV)
    assert "ok" in r.stdout


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm toolchain missing")
def test_library_host_code_under_asan_and_ubsan(tmp_path):
    objs = []
    for f in sorted(os.listdir(CSRC)):
        if not f.endswith((".hip", ".cpp")):
            continue
        o = str(tmp_path / (f + ".o"))
        host_san = [a for flag in SAN_FLAGS for a in ("-Xarch_host", flag)]
        _run([HIPCC, "-x", "hip", "--offload-host-only", "-O1", "-g", "-std=c++17", "-fPIC",
              "-I", os.path.join(ROOT, "include"), "-I", CSRC, *host_san, "-w",
              "-c", os.path.join(CSRC, f), "-o", o])
        objs.append(o)
    # the host-only objects name their (absent) device code objects
    undef = _run(["nm", "-u", *objs]).stdout
    fat = sorted(set(re.findall(r"\b(__hip_fatbin_[0-9a-f]+)\b", undef)))
    stub_fat = tmp_path / "fatbins.c"
    stub_fat.write_text("".join(f"char {s}[16];\n" for s in fat))
    exe = str(tmp_path / "host_checks")
    _run([CLANG, "-O1", "-g", *SAN_FLAGS, "-I", os.path.join(ROOT, "include"), "-o", exe,
          os.path.join(SAN, "host_checks.c"), os.path.join(SAN, "hip_stub.c"), str(stub_fat), *objs,
          "-lstdc++", "-lm", "-lpthread"])
    r = _run([exe], env=ENV)
    assert "launches" in r.stdout
    print(r.stdout)
