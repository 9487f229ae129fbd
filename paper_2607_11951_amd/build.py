"""Builds libgrid.so in-tree: host C++ with g++, kernels with hipcc for gfx950."""

import os
import subprocess
from pathlib import Path

PKG = Path(__file__).resolve().parent
CSRC = PKG / "csrc"
OUT = PKG / "libgrid.so"
BUILD = PKG / "_build"
HOST_SOURCES = ["grammar.cpp", "lexer.cpp", "parser.cpp", "artifacts.cpp", "advance.cpp", "complete.cpp", "capi.cpp"]
HIP_SOURCES = ["kernels.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-pthread", "-Wall", "-Wextra", "-Wno-unused-parameter"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(str(c) for c in cmd), flush=True)
    subprocess.run([str(c) for c in cmd], check=True)


def build(verbose=False, jobs=8):
    BUILD.mkdir(exist_ok=True)
    objs = []
    procs = []
    for src in HOST_SOURCES:
        obj = BUILD / (src + ".o")
        cmd = ["g++", *HOST_FLAGS, "-c", CSRC / src, "-o", obj]
        if verbose:
            print(" ".join(str(c) for c in cmd), flush=True)
        procs.append(subprocess.Popen([str(c) for c in cmd]))
        objs.append(obj)
    for src in HIP_SOURCES:
        obj = BUILD / (src + ".o")
        cmd = [HIPCC, *HIP_FLAGS, "-c", CSRC / src, "-o", obj]
        if verbose:
            print(" ".join(str(c) for c in cmd), flush=True)
        procs.append(subprocess.Popen([str(c) for c in cmd]))
        objs.append(obj)
    bad = [p.args for p in procs if p.wait() != 0]
    if bad:
        raise RuntimeError(f"compile failed: {bad}")
    tmp = str(OUT) + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-pthread", "-o", tmp, *objs], verbose)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
