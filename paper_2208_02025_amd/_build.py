"""Build libollie.so (the gfx950 HIP library behind include/ollie.h) with hipcc.

Each .hip source is compiled for gfx950 only, then linked into one shared library
next to this file.  Run ``python -m paper_2208_02025_amd._build`` or call build().

Next to the library the build writes ``libollie.so.sha256``: a digest of every input
of the build (sources, headers, flags).  The loader rebuilds when the digest of the
sources on disk differs from it, so a stale binary is never used silently.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import hashlib
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OBJ_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libollie.so")
STAMP = LIB + ".sha256"
HEADER = os.path.join(os.path.dirname(HERE), "include", "ollie.h")
SOURCES = ["abi.hip", "gemm.hip", "eop.hip", "band.hip", "conv_fused.hip", "split3.hip"]
ARCH = "gfx950"

# Packed fp32 ops are disabled for all device code (the host pass warns that it does
# not know the feature; that is harmless).  Symbols are hidden by default; abi.hip
# exports exactly the functions include/ollie.h declares.
HIPCC_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", f"--offload-arch={ARCH}",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Wall", "-Wno-unused-function"]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the ROCm toolchain is required to build libollie.so")


# Per-source extra flags.  The large fused-convolution tiles keep 96 accumulator
# registers per lane live next to two operand-fragment sets; the VGPR form of the MFMA
# keeps them in place (with accumulators in AGPRs the register allocator shuffled them
# between the two register files every iteration).
SOURCE_FLAGS = {"conv_fused.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def source_digest(csrc: str = CSRC, header: str = HEADER) -> str:
    """sha256 over the build inputs: every file under csrc/, the public header and the
    compiler flags (in a fixed order)."""
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(csrc, "*")))
    for f in files + [header]:
        h.update(os.path.basename(f).encode() + b"\0")
        with open(f, "rb") as fh:
            h.update(fh.read())
        h.update(b"\0")
    h.update(repr((SOURCES, HIPCC_FLAGS, sorted(SOURCE_FLAGS.items()), ARCH)).encode())
    return h.hexdigest()


def is_current(lib: str = LIB, stamp: str = STAMP) -> bool:
    """True when `lib` exists and was built from the sources now on disk."""
    if not (os.path.exists(lib) and os.path.exists(stamp)):
        return False
    with open(stamp) as fh:
        return fh.read().strip() == source_digest()


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(OBJ_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [_hipcc(), *HIPCC_FLAGS, *SOURCE_FLAGS.get(src, []), "-c", os.path.join(CSRC, src),
           "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{res.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    digest = source_digest()
    os.makedirs(OBJ_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, LIB)
    with open(STAMP + ".tmp", "w") as fh:
        fh.write(digest + "\n")
    os.replace(STAMP + ".tmp", STAMP)
    return LIB


def asan_runtime() -> str:
    """The clang AddressSanitizer runtime that a process loading build_sanitized()'s
    library must preload (the library itself does not link it)."""
    res = subprocess.run([os.path.join(os.path.dirname(_hipcc()), "..", "llvm", "bin", "clang"),
                          "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True)
    path = res.stdout.strip()
    if res.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError("clang AddressSanitizer runtime not found")
    return path


def build_sanitized(out_dir: str, verbose: bool = False) -> str:
    """A copy of the library whose host code in abi.hip (argument validation, sizing,
    dispatch) is built with AddressSanitizer and UndefinedBehaviorSanitizer; device
    code is built as usual, and the other sources are the regular objects.  For CPU
    tests of the host logic; load it with asan_runtime() preloaded."""
    if not all(os.path.exists(os.path.join(OBJ_DIR, os.path.splitext(s)[0] + ".o"))
               for s in SOURCES):
        build(verbose)
    os.makedirs(out_dir, exist_ok=True)
    obj = os.path.join(out_dir, "abi_san.o")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
    cmd = [_hipcc(), *HIPCC_FLAGS, *san, "-c", os.path.join(CSRC, "abi.hip"), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on abi.hip (sanitized):\n{res.stderr}")
    objs = [obj] + [os.path.join(OBJ_DIR, os.path.splitext(s)[0] + ".o")
                    for s in SOURCES if s != "abi.hip"]
    lib = os.path.join(out_dir, "libollie_san.so")
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Xarch_host",
           "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-o", lib, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed (sanitized):\n{res.stderr}")
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
