"""The host-side C++ of the library (plan bookkeeping, argument checks, the
offline clustering and rank allocation) under AddressSanitizer and
UndefinedBehaviorSanitizer: the host tests run again, in a subprocess,
against the sanitized build (paper_2607_24331_amd/build.py --sanitize, also
made by __graft_entry__.build()), with the sanitizer runtime preloaded; any
report aborts that run."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2607_24331_amd", "libdckv_sanitized.so")


def _asan_runtime():
    try:
        path = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True,
                              check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(not os.path.exists(LIB), reason="sanitized library not built (build.py --sanitize)")
def test_host_code_under_asan_and_ubsan():
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("no AddressSanitizer runtime for g++")
    env = dict(os.environ, DCKV_LIBRARY=LIB, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_lib_host.py"),
                        os.path.join(ROOT, "tests", "test_lib_offline_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in tail and "runtime error" not in tail, tail
