"""The library's host logic under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): build _build/liblp_san.so, whose host-side translation units are
instrumented, and run the C-ABI host tests against it in a child process with
the sanitizer runtime preloaded. Any report (out-of-bounds access, use after
free, undefined behaviour) aborts the child and fails this test."""
import os
import subprocess
import sys

import pytest

from paper_1812_04352_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_logic_is_clean_under_sanitizers():
    rt = B.sanitizer_runtime()
    if not os.path.exists(rt):
        pytest.skip("no AddressSanitizer runtime in this toolchain")
    lib = B.build_sanitized(verbose=False)
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, LP_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in out, out[-4000:]
    assert "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in r.stdout
