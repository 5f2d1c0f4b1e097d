"""The oracle and the library's host-side logic under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

Both are rebuilt with the sanitizers into a temporary directory, then the oracle pins
(tests/test_oracle_pins.py) and the C ABI checks (tests/test_abi_cpu.py: argument
validation, sizing, the exported symbols) run in child processes that load those
builds, with the matching sanitizer runtime preloaded (gcc's for the oracle, clang's
for the library).  A sanitizer report aborts the child, so the test fails on any
out-of-bounds access, use-after-free or undefined behaviour those tests reach.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ASAN_OPTS = "detect_leaks=0:abort_on_error=1:halt_on_error=1:alloc_dealloc_mismatch=0"


def _run(env_extra, args):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = ASAN_OPTS
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                           *args], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=900)


def test_oracle_pins_under_asan_ubsan(tmp_path):
    from oracle import build as ob
    lib = ob.build_sanitized(str(tmp_path))
    res = _run({"OLLIE_ORACLE_LIBRARY": lib, "LD_PRELOAD": ob.asan_runtime(),
                "OMP_NUM_THREADS": "4"},
               ["tests/test_oracle_pins.py", "-m", "not gpu"])
    assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
    assert " passed" in res.stdout


def test_abi_host_checks_under_asan_ubsan(tmp_path):
    from paper_2208_02025_amd import _build
    try:
        lib = _build.build_sanitized(str(tmp_path))
        rt = _build.asan_runtime()
    except RuntimeError as e:   # no ROCm toolchain: nothing to build the library with
        pytest.skip(str(e))
    res = _run({"OLLIE_LIBRARY": lib, "LD_PRELOAD": rt},
               ["tests/test_abi_cpu.py", "-m", "not gpu", "-k",
                "not stale_library and not build_digest"])
    assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
    assert " passed" in res.stdout
