"""The host-side C ABI checks (tests/test_abi_cpu.py: size queries, argument
validation, error paths; no kernel launch) against a build of the library whose
host code (api.hip, the host eigensolver) carries AddressSanitizer and
UndefinedBehaviorSanitizer, any report fatal, in a child process that preloads
clang's ASan runtime."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _clang_asan():
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def test_abi_checks_under_asan_and_ubsan():
    rt = _clang_asan()
    if rt is None:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    from paper_2609_26425_amd import build
    lib = build.build_sanitized()
    env = dict(os.environ, QWM_LIB=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:alloc_dealloc_mismatch=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    p = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_cpu.py"), "-x", "-q",
                        "-p", "no:cacheprovider", "-k", "not xcd"], env=env, cwd=ROOT, capture_output=True, text=True,
                       timeout=900)
    tail = (p.stdout + p.stderr)[-3000:]
    assert p.returncode == 0, tail
    assert "passed" in p.stdout and "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
