"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU, no GPU): tests/host/abi_host_check.cpp drives the C ABI's size queries,
configuration and argument validation, error strings, null handles, the
allocation-free remap's and the probes' argument checks, and wam_init
failing cleanly; any memory error or undefined behaviour aborts the run."""
import os
import subprocess

import pytest


@pytest.mark.slow
def test_host_abi_under_sanitizers():
    from paper_2609_34608_amd import build
    if not os.path.exists(build.HIPCC) or not os.path.exists(build.CLANGXX):
        pytest.skip("ROCm toolchain not present")
    exe = build.build_host_check()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "host ABI checks passed" in r.stdout
