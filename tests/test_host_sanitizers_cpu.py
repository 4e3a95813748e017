"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

A build of libasrkf.so whose host part (configuration checks, context set-up,
the ABI's argument validation, the Eq. 3 table) is instrumented runs the host
ABI checks of test_abi_cpu.py in a child process with the sanitizer runtime
preloaded; any report ends that process with an error.  No GPU is needed: the
calls exercised here return before any device work.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def test_abi_checks_under_address_and_ub_sanitizers(tmp_path):
    if os.environ.get("LD_PRELOAD"):
        pytest.skip("a library is already preloaded into this process tree; not replacing it")
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("clang AddressSanitizer runtime not found")
    sys.path.insert(0, os.path.join(ROOT, "paper_2512_11221_amd"))
    import build as lib_build
    lib = lib_build.build_sanitized(("address", "undefined"), out=str(tmp_path / "libasrkf_san.so"))
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, ASRKF_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider", os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, (r.stdout[-3000:] + r.stderr[-3000:])
    assert "passed" in r.stdout
