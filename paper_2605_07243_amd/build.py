"""Build libspecblock.so for gfx950 with hipcc (in-tree).

    python -m paper_2605_07243_amd.build
"""
from __future__ import annotations

import os
import shlex
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libspecblock.so")
SOURCES = ["gemm.hip", "elementwise.hip", "attention.hip", "vocab.hip",
           "tree.hip", "sampling.hip", "adapt.hip",
           "engine.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
         # packed fp32 VALU forms are kept out of the generated code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed: " + " ".join(cmd) + "\n" + r.stdout
                           + r.stderr)
    return r


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link the shared library; returns its
    path.  Always rebuilds."""
    os.makedirs(BUILD, exist_ok=True)

    def one(src):
        obj = os.path.join(BUILD, src + ".o")
        cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        _run(cmd)
        return obj

    with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(one, SOURCES))
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o",
          tmp])
    os.replace(tmp, LIB)
    return LIB


ASAN_LIB = os.path.join(BUILD, "asan", "libspecblock_asan.so")


def build_host_asan(verbose: bool = False) -> str:
    """The same library with AddressSanitizer on its host code only (device
    code is built as usual); loading it needs the clang ASan runtime
    preloaded.  For the CPU checks of the host-side ABI paths."""
    out = os.path.dirname(ASAN_LIB)
    os.makedirs(out, exist_ok=True)
    san = shlex.split("-Xarch_host -fsanitize=address "
                      "-Xarch_host -fno-omit-frame-pointer")

    def one(src):
        obj = os.path.join(out, src + ".o")
        cmd = [HIPCC, *FLAGS, *san, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        _run(cmd)
        return obj

    with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(one, SOURCES))
    tmp = ASAN_LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o",
          tmp])
    os.replace(tmp, ASAN_LIB)
    return ASAN_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
