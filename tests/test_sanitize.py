"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer: the
library's offline pack / unpack (quick_pack.cpp) and the CPU oracle
(oracle/oracle.c), built with -fsanitize=address,undefined by the host
compilers (no GPU code involved) and driven by tests/sanitize_main.c on
exactly-sized buffers.  Any out-of-bounds access, use after free, leak or
undefined arithmetic aborts the driver."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _have(tool):
    return shutil.which(tool) is not None


@pytest.mark.skipif(not (_have("gcc") and _have("g++")), reason="host compilers not found")
def test_pack_and_oracle_under_sanitizers(tmp_path):
    inc = os.path.join(ROOT, "include")
    csrc = os.path.join(ROOT, "paper_2402_10076_amd", "csrc")
    objs = []
    steps = [
        (["g++", "-std=c++17", "-pthread", "-I", inc, "-I", csrc] + SAN,
         os.path.join(csrc, "quick_pack.cpp"), "pack.o"),
        (["gcc", "-std=c11", "-fopenmp"] + SAN, os.path.join(ROOT, "oracle", "oracle.c"), "oracle.o"),
        (["gcc", "-std=c11", "-I", inc] + SAN, os.path.join(ROOT, "tests", "sanitize_main.c"), "main.o"),
    ]
    for cmd, src, obj in steps:
        out = str(tmp_path / obj)
        r = subprocess.run(cmd + ["-c", src, "-o", out], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        objs.append(out)
    exe = str(tmp_path / "sanitize_main")
    r = subprocess.run(["g++", "-fopenmp", "-pthread"] + SAN + objs + ["-o", exe, "-lm"], capture_output=True,
                       text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and "SANITIZE_OK" in r.stdout, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
