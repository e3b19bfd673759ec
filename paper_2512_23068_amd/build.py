"""Builds libpgf.so (the HIP library) in-tree for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(_HERE)
CSRC = os.path.join(_HERE, "csrc")
OUT = os.path.join(_HERE, "libpgf.so")
SOURCES = ["pgf_scan.hip", "pgf_scan_f32.hip", "pgf_scan_bf16.hip", "pgf_la.hip", "pgf_plan.cpp", "pgf_timing.cpp",
           "pgf_stream.cpp"]
# Packed FP32 instructions stay disabled in every HIP object of this library.
HIPCC_FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Wall", "-Wno-unused-function"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return "hipcc"


def build(verbose: bool = False) -> str:
    """Compiles every source to an object in parallel, links libpgf.so."""
    objdir = os.path.join(ROOT, "_build")
    os.makedirs(objdir, exist_ok=True)
    procs, objs = [], []
    for src in SOURCES:
        obj = os.path.join(objdir, src + ".o")
        cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), "-c", os.path.join(CSRC, src),
               "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = "\n".join(l for l in out.decode(errors="replace").splitlines()
                         if "packed-fp32-ops" not in l)
        if p.returncode != 0:
            failed.append(src)
            sys.stderr.write(text + "\n")
        elif verbose and text.strip():
            print(text)
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    tmp = OUT + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    subprocess.run(cmd, check=True)
    os.replace(tmp, OUT)
    return OUT


CALLER_SRC = os.path.join(ROOT, "tests", "native", "pgf_c_caller.cpp")
CALLER = os.path.join(ROOT, "tests", "native", "pgf_c_caller")


def build_caller() -> str:
    """Compiles the plain C-ABI caller used by the tests (host code only),
    linked against the in-tree libpgf.so."""
    tmp = CALLER + ".tmp"
    cmd = [hipcc(), "-O2", "-std=c++17", "--offload-arch=gfx950", "-I", os.path.join(ROOT, "include"), CALLER_SRC,
           "-o", tmp, "-L", _HERE, "-lpgf", "-Wl,-rpath,$ORIGIN/../../paper_2512_23068_amd"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, CALLER)
    return CALLER


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_caller())
