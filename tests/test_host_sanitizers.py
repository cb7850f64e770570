"""The library's host code (argument validation, workspace sizing, the
schedule and Eq. psaw helpers, dispatch up to the launch) under
AddressSanitizer and UndefinedBehaviorSanitizer: a host-instrumented build
of libprhs runs the whole host ABI suite in a child process with the ASan
runtime preloaded; any report aborts the child."""

import glob
import os
import subprocess
import sys

import pytest

from paper_2602_08329_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = """
import sys
sys.path.insert(0, {root!r})
import paper_2602_08329_amd.binding as B
B.LIB_PATH = {lib!r}
import pytest
sys.exit(pytest.main(["-q", "-x", "-p", "no:cacheprovider", {tests!r}]))
"""


def test_host_abi_suite_under_asan_and_ubsan(tmp_path):
    rts = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rts:
        pytest.skip("no clang ASan runtime in this image")
    lib = build.build(host_sanitize=str(tmp_path / "libprhs_san.so"))
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms, "the build is not instrumented"
    env = dict(os.environ, LD_PRELOAD=rts[-1],
               ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    code = CHILD.format(root=ROOT, lib=lib, tests=os.path.join(ROOT, "tests", "test_abi_host.py"))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600, cwd=ROOT)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in tail, tail
