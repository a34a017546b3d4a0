"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

tests/sanitize/build.sh compiles every library source with both sanitizers on the host code
and links tests/sanitize/abi_validation.cpp, which drives a validation-only context through
every argument check, the network validator (fixed cases, extreme sizes, seeded random node
lists) and both planners.  Any sanitizer report aborts the program."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC) or shutil.which("bash") is None, reason="needs hipcc")
def test_abi_validation_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "abi_validation")
    b = subprocess.run(["bash", os.path.join(HERE, "sanitize", "build.sh"), exe], capture_output=True, text=True)
    assert b.returncode == 0, b.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, "3000"], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "all checks passed" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
