"""Builds libsparrow.so (gfx950) in-tree with hipcc.

``python -m paper_2606_08446_amd.build`` or ``build_library()``.  Every call
recompiles.  Objects go to ``paper_2606_08446_amd/_build`` (not committed).
``--sanitize`` builds ``libsparrow_asan.so`` instead, its host code (argument
checks, workspace sizing, the host-side budget bound, launch set-up) with
AddressSanitizer and UndefinedBehaviorSanitizer; the device code is unchanged.
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
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsparrow.so")
SOURCES = ["api.hip", "meta.hip", "append.hip", "score_topk.hip", "attention.hip",
           "acceptance.hip", "measure.hip"]
ARCH = "gfx950"
# Packed fp32 VALU ops are switched off for every device compile.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
CFLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          "-I", INCLUDE, "-I", CSRC] + DEVICE_FLAGS


def hipcc() -> str:
    for c in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), "hipcc"):
        if os.path.sep not in c or os.path.exists(c):
            return c
    return "hipcc"


# Host-side sanitizers: every -fsanitize= is preceded by -Xarch_host, so only the host
# compilation is instrumented.
SANITIZE_FLAGS = ["-g", "-fno-omit-frame-pointer", "-Xarch_host", "-fsanitize=address",
                  "-Xarch_host", "-fsanitize=undefined"]
LIB_ASAN = os.path.join(PKG, "libsparrow_asan.so")


def _compile(src: str, sanitize: bool = False) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ("_asan.o" if sanitize else ".o"))
    cmd = [hipcc()] + CFLAGS + (SANITIZE_FLAGS if sanitize else []) + \
        ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build_library(verbose: bool = False, sanitize: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda src: _compile(src, sanitize), SOURCES))
    lib = LIB_ASAN if sanitize else LIB
    tmp = lib + ".tmp"
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    if sanitize:
        cmd += ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print("built", lib)
    return lib


if __name__ == "__main__":
    build_library(verbose=True, sanitize="--sanitize" in sys.argv[1:])
    sys.exit(0)
