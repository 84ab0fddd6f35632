"""The host side of the C ABI (argument validation, handle and workspace
bookkeeping, the launch sequences' host code) built with AddressSanitizer,
and the ABI checks of test_abi.py run against that build in a child process
that preloads the ASan runtime.  CPU only: every check there fails before
any HIP call."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc is needed to build the ASan library")
def test_abi_checks_pass_under_host_asan():
    from paper_2608_02438_amd import build as b
    lib = b.build(asan=True)
    out = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True)
    assert "__asan_report" in out.stdout, "the library is not instrumented"
    env = dict(os.environ, XPRESS_LIB=lib, LD_PRELOAD=b.asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "AddressSanitizer" not in r.stderr
