"""Host-side memory and undefined-behaviour checks of the library.

Every source of the library is compiled for the host alone with
AddressSanitizer and UndefinedBehaviorSanitizer and linked against a stub HIP
runtime (host memory as device memory, launches that run nothing); a driver
then calls every entry point of the C ABI over the option space, with every
documented argument error and the staged calls in and out of order.  Kernel
arithmetic is covered by the GPU parity tests; this covers the host code
around it: argument checks, workspace layouts, tile and task lists, launch
geometry, error paths.
"""
import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "host_sanitize"))


@pytest.mark.skipif(not (shutil.which("hipcc") or os.path.exists("/opt/rocm/bin/hipcc")),
                    reason="hipcc is needed to compile the library's host code")
def test_abi_under_address_and_ub_sanitizers(tmp_path):
    import build as host_build
    exe = host_build.build(str(tmp_path))
    env = dict(os.environ, ASAN_OPTIONS="abort_on_error=1:detect_leaks=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "checks passed" in r.stdout
    assert "runtime error" not in out and "ERROR: AddressSanitizer" not in out
