"""The host code of the library under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU): the planner, the block manager and the
validation of the C ABI are rebuilt with both sanitizers
(build.build_sanitized) and the host-only test files run against that build
in a child interpreter with the sanitizer runtime preloaded; any report
aborts the child.  (No GPU: every call in those files is host-only or fails
validation before any launch.)"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST_TESTS = ["tests/test_plan_invariants.py", "tests/test_kvm.py", "tests/test_abi_host.py"]


@pytest.mark.slow
def test_host_code_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    from paper_2504_03651_amd import build
    lib = build.build_sanitized(out=str(tmp_path / "libecho_san.so"))
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms, "not an instrumented build"
    env = dict(os.environ, ECHO_LIBRARY=lib, LD_PRELOAD=build.sanitizer_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *HOST_TESTS], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=900)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
