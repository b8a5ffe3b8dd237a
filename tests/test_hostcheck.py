"""The ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/test_abi.py (every export, every validation path, no GPU needed) runs
in a child process against a library whose host code is instrumented
(tests/hostcheck_build.py); any sanitizer report ends that process with an
error.  Skipped when the ASan runtime or the normal build's kernel objects
are missing.
"""

import os
import subprocess
import sys

import pytest

import hostcheck_build as H

pytestmark = pytest.mark.skipif(H.asan_runtime() is None or H.kernel_objects() is None,
                                reason="needs the ROCm clang ASan runtime and a normal build")

RUNNER = """
import sys
import paper_2402_00518_amd.binding as B
B.LIB_PATH = sys.argv[1]
import pytest
sys.exit(pytest.main(["-q", "-s", "-p", "no:cacheprovider", sys.argv[2]]))
"""


def test_abi_validation_under_asan_and_ubsan(tmp_path):
    lib = H.build(str(tmp_path))
    env = dict(os.environ, LD_PRELOAD=H.asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", RUNNER, lib, os.path.join(H.ROOT, "tests", "test_abi.py")],
                       cwd=H.ROOT, env=env, capture_output=True, text=True, timeout=600)
    report = (r.stdout + r.stderr)[-4000:]
    assert "Sanitizer" not in r.stderr, report
    assert r.returncode == 0, report
    assert " passed" in r.stdout, report
