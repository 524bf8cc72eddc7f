"""The C-ABI layer (argument validation, workspace carve-up, dispatch) under
AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

build.py compiles csrc/aal_api.hip with the host sanitizers; this test links
it with host-only stand-ins for the kernel launchers (tests/sanitize/
launch_stubs.cpp, which write every byte of the workspace regions the kernels
would use) and a driver that calls every entry point with valid and invalid
arguments (tests/sanitize/abi_driver.cpp), then runs it.  Workspaces are host
buffers of exactly the advertised size, so any carve-up past the end is a
heap-buffer-overflow report; enum arguments outside their enumerators and
other undefined behaviour abort the run.  No GPU is needed."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")


def test_abi_layer_under_asan_and_ubsan(tmp_path):
    from paper_2609_24150_amd import build as B
    try:
        hipcc = B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not found")
    obj = B.compile_api_sanitized(str(tmp_path / "aal_api_asan.o"))
    exe = tmp_path / "abi_sanitize"
    cmd = [hipcc, "-std=c++17", f"--offload-arch={B.ARCH}", *B.SANITIZE_FLAGS, f"-I{B.INCLUDE}", f"-I{B.CSRC}",
           obj, os.path.join(SAN, "launch_stubs.cpp"), os.path.join(SAN, "abi_driver.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "all checks passed" in r.stdout
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
