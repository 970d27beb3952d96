"""The C-ABI host layer under AddressSanitizer and UndefinedBehaviorSanitizer.

The argument checks, workspace arithmetic and struct handling of api.cpp are
compiled by g++ with both sanitizers (build.build_host_sanitized) and the
host-side ABI tests run against that library in a child process, so that an
out-of-bounds access, use after free, overflow or other undefined behaviour
on any validation path aborts the run.  No kernel is launched."""

import os
import subprocess
import sys

from paper_2608_15018_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_checks_pass_under_host_sanitizers():
    lib = build.build_host_sanitized(verbose=False)
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    assert "__asan_" in syms and "__ubsan_" in syms     # really instrumented
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       cwd=ROOT, env=build.host_sanitizer_env(), capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert " passed" in r.stdout and "failed" not in r.stdout
