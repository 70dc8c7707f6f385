"""Builds libspla.so (HIP, gfx950) and libspla_host.so (host-only checks).

    python -m paper_2601_22379_amd.build [--jobs N] [--verbose]

Every translation unit is compiled with hipcc for gfx950 into _build/, then
linked into paper_2601_22379_amd/libspla.so next to this file. The host-only
part of the C ABI (validation and sizing) is also built with g++ into
libspla_host.so, which loads on machines without a GPU or HIP runtime.
"""

from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libspla.so")
HOST_LIB = os.path.join(PKG, "libspla_host.so")
ARCH = os.environ.get("SPLA_OFFLOAD_ARCH", "gfx950")

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Wno-unused-function", "-Wno-unused-variable",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def sources() -> list:
    out = []
    for f in sorted(os.listdir(CSRC)):
        if f.endswith(".hip") or f.endswith(".cpp"):
            out.append(os.path.join(CSRC, f))
    return out


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}")
    return r


def build(jobs: int = 8, verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    objs = []
    cmds = []
    for src in sources():
        obj = os.path.join(BUILD, os.path.basename(src) + ".o")
        objs.append(obj)
        lang = ["-x", "hip"]
        cmds.append([hipcc, *lang, *HIP_FLAGS, "-c", src, "-o", obj])
    with ThreadPoolExecutor(max(1, jobs)) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    build_host(verbose)
    return LIB


def build_host(verbose: bool = False) -> str:
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        raise RuntimeError("no host C++ compiler found")
    tmp = HOST_LIB + ".tmp"
    _run([cxx, "-std=c++17", "-O2", "-Wall", "-Wextra", "-fPIC", "-shared",
          "-I", os.path.join(ROOT, "include"), os.path.join(CSRC, "spla_host.cpp"), "-o", tmp],
         verbose)
    os.replace(tmp, HOST_LIB)
    return HOST_LIB


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=min(8, os.cpu_count() or 1))
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--host-only", action="store_true")
    a = ap.parse_args(argv)
    print(build_host(a.verbose) if a.host_only else build(a.jobs, a.verbose))


if __name__ == "__main__":
    main()
