"""Build libdlm.so (the HIP kernels and the C ABI) for gfx950 with hipcc, and
libdlmctl.so (the host-only threshold controller) with g++.

Usage: python -m paper_2606_29094_amd.build  (or call build()).
Every call recompiles; objects go to _build/ next to the package.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libdlm.so")
CTL_OUT = os.path.join(PKG, "libdlmctl.so")
BUILD = os.path.join(os.path.dirname(PKG), "_build", "dlm")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = ["runtime.hip", "gemm.hip", "gemm_dl.hip", "rowwise.hip", "attention.hip", "ceiling.hip"]
FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-result"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("command failed: %s\n%s" % (" ".join(cmd), err))
    return err


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []

    def one(src):
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        err = _run([HIPCC, *FLAGS, "-I", SRC, "-c", os.path.join(SRC, src), "-o", obj])
        if verbose and err.strip():
            print(err, file=sys.stderr)
        return obj

    jobs = int(os.environ.get("MAX_JOBS", "8"))
    with ThreadPoolExecutor(max_workers=min(jobs, len(SOURCES))) as ex:
        objs = list(ex.map(one, SOURCES))
    tmp = OUT + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, OUT)
    build_controller()
    return OUT


def build_controller() -> str:
    tmp = CTL_OUT + ".tmp"
    _run(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-Wall", "-Wextra", "-o", tmp,
          os.path.join(SRC, "controller.cpp")])
    os.replace(tmp, CTL_OUT)
    return CTL_OUT


if __name__ == "__main__":
    print(build(verbose=True))
