"""Build the HIP library libquick.so in-tree for gfx950 (hipcc cross-compiles
without a GPU).  quick_gemm.hip is compiled as three translation units in
parallel (host code and the C ABI; the stream-kernel launches; the
tiled-kernel launches), then linked with the packing code."""
from __future__ import annotations

import os
import subprocess
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libquick.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# -packed-fp32-ops: keep the compiler from emitting packed fp32 VALU ops.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-pthread",
         "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]
# (source, extra flags) of each translation unit
UNITS = [("quick_pack.cpp", []),
         ("quick_gemm.hip", ["-DQUICK_PART=0"]),
         ("quick_gemm.hip", ["-DQUICK_PART=1"]),
         ("quick_gemm.hip", ["-DQUICK_PART=2"])]


def _msgs(r):
    return [l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l or "error" in l]


def build(verbose: bool = False, extra=()) -> str:
    with tempfile.TemporaryDirectory(prefix="quick_build_") as tmpd:
        procs = []
        for i, (src, fl) in enumerate(UNITS):
            obj = os.path.join(tmpd, "u%d.o" % i)
            cmd = [HIPCC] + FLAGS + fl + list(extra) + ["-c", "-o", obj, os.path.join(CSRC, src)]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((obj, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)))
        objs, out, failed = [], [], False
        for obj, p in procs:
            so, se = p.communicate()
            r = subprocess.CompletedProcess(p.args, p.returncode, so, se)
            out += _msgs(r)
            failed |= p.returncode != 0
            objs.append(obj)
        if failed:
            raise RuntimeError("hipcc failed:\n" + "\n".join(out))
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-pthread", "-o", tmp] + objs
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        out += _msgs(r)
        if r.returncode != 0:
            raise RuntimeError("link failed:\n" + "\n".join(out))
    if verbose and out:
        print("\n".join(out))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
