"""The C-ABI validation, the host planners and the block's host code under
AddressSanitizer and UndefinedBehaviorSanitizer: api.cpp, plan.cpp and
block.cpp rebuilt with host-side sanitizers (paper_2404_19429_amd/build.py,
build_host_sanitized), and the CPU tests of the ABI and of the planners run
against that library in a child process with the sanitizer runtime preloaded
(any report aborts the child)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2404_19429_amd import build as B  # noqa: E402


def test_abi_and_planner_tests_pass_under_asan_and_ubsan():
    if not all(os.path.exists(os.path.join(B.BUILD, os.path.splitext(s)[0] + ".o"))
               for s in B.SOURCES if s not in B.SANITIZED_SOURCES):
        pytest.skip("the regular build's objects are missing (run the build first)")
    lib = B.build_host_sanitized()
    rt = B.asan_runtime()
    assert os.path.exists(rt), rt
    env = dict(os.environ, LD_PRELOAD=rt, LANCET_MOE_LIB=lib, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "tests/test_abi_cpu.py", "tests/test_dw_schedule.py", "-q",
                        "-m", "not gpu", "-p", "no:cacheprovider", "-x"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
