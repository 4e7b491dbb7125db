"""The host layer under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only): every source is rebuilt with both sanitizers on the host code (the
argument checks, sizing and launch set-up of the C ABI), and the C-ABI
argument tests of test_abi.py run against that build in a child process with
the sanitizer runtime preloaded.  Any sanitizer report aborts the child
(UB checks do not recover), so a clean exit means no report."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs hipcc to build the sanitized host layer")
def test_abi_checks_clean_under_asan_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2609_23153_amd import build as B
    lib = B.build_host_sanitized()
    env = dict(os.environ)
    env["SPARSE_ATTN_LIB"] = lib
    env["LD_PRELOAD"] = B.asan_runtime()
    # Python itself is not instrumented: its allocations look like leaks
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
