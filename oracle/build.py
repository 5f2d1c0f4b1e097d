"""Compile the CPU oracle (oracle.c) into liboracle.so with gcc and OpenMP.

Test infrastructure only.  No -ffast-math: sums keep the order the source states.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall",
           "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_sanitized(out_dir: str, verbose: bool = False) -> str:
    """liboracle built with AddressSanitizer and UndefinedBehaviorSanitizer (gcc), for
    CPU test runs with gcc's libasan preloaded (see asan_runtime())."""
    os.makedirs(out_dir, exist_ok=True)
    lib = os.path.join(out_dir, "liboracle_san.so")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall",
           "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           "-fno-sanitize-recover=all", "-o", lib, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return lib


def asan_runtime() -> str:
    """gcc's AddressSanitizer runtime, to preload into a process that loads
    build_sanitized()'s library."""
    out = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                         text=True, check=True).stdout.strip()
    if not os.path.isabs(out) or not os.path.exists(out):
        raise RuntimeError("gcc AddressSanitizer runtime not found")
    return os.path.realpath(out)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
