"""The library's host code (layout validation and tables, the state machine,
the persistence store's manifest parsing, crash repair and writer pool)
under AddressSanitizer and UndefinedBehaviorSanitizer: the CPU tests of the
interface and of the store run in a child process against the sanitized
build, with the sanitizer runtime preloaded; any report fails the run."""
import os
import subprocess
import sys

import pytest

from paper_2609_27193_amd.build_lib import SANITIZED_LIB, sanitizer_runtime

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_cpu_interface_tests_under_host_sanitizers():
    rt = sanitizer_runtime()
    if not os.path.exists(SANITIZED_LIB) or not rt:
        pytest.skip("the host-sanitized library is built by __graft_entry__.build()")
    env = dict(os.environ, LD_PRELOAD=rt, LAYERCHECK_LIB=SANITIZED_LIB,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        "tests/test_abi.py", "tests/test_store.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error:" not in tail, tail
