"""Build libcmc.so (the HIP library behind include/cmc.h) for gfx950.

Each HIP source is compiled by hipcc in parallel, then linked into a shared
library inside the package directory, so it ships with the source tree.
Packed fp32 instructions are disabled for every HIP translation unit.
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "libcmc.so")
OBJDIR = os.path.join(PKG, "_build")
SOURCES = ["cmc_api.hip", "decode.hip", "select.hip", "window.hip", "denoise.hip", "bridge.hip"]
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE, "-I", CSRC,
         # Leading scalar kernel arguments arrive in SGPRs at wave launch (the
         # decode kernel passes the fields its first loads need that way).
         "-mllvm", "-amdgpu-kernarg-preload-count=14"]


def _compile(src: str, objdir: str = OBJDIR, defines=()) -> str:
    obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *[f"-D{d}" for d in defines], "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False, output: str = LIBRARY, defines=()) -> str:
    """Compile every HIP source and link the library (libcmc.so in the
    package by default); `defines` are NAME=VALUE build-time tuning knobs.
    Returns the library path."""
    objdir = OBJDIR if output == LIBRARY else output + ".objs"
    os.makedirs(objdir, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda src: _compile(src, objdir, defines), SOURCES))
    tmp = output + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, output)
    if verbose:
        print(f"built {output}")
    return output


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
