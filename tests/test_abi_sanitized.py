"""The C-ABI checks of ``test_abi.py`` run again against a build of the
library whose host code carries AddressSanitizer and UndefinedBehaviorSanitizer
(argument validation, layout sizing, workspace and launch planning all run on
the host).  Any invalid memory access or undefined behaviour in that code
aborts the child process and fails this test.  CPU only: every call in
``test_abi.py`` is rejected before the library makes a HIP call."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.slow
def test_abi_checks_under_host_sanitizers():
    from paper_2606_11357_amd import sanitized_build
    lib = sanitized_build.build_sanitized()
    env = dict(os.environ)
    env.update({
        "TILEFUSE_LIB": lib,
        "LD_PRELOAD": sanitized_build.runtime(),
        # the interpreter's own allocations are not the subject (and are
        # never freed at exit)
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
    })
    # test_binding_refuses_cpu_tensors imports torch, whose own libraries
    # are not built for the sanitizer's interposed allocator
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py"), "-k", "not binding_refuses"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert " passed" in r.stdout and "failed" not in r.stdout
