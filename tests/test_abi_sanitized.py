"""The host-side ABI tests again, against a build of the library whose host code
(argument validation, the plan registry, workspace layout) is compiled with
AddressSanitizer and UndefinedBehaviorSanitizer (undefined behaviour traps).

The sanitized library is built by paper_2106_12736_amd.build.build_host_sanitized
(device objects shared with the normal build) and loaded in a child process with
the sanitizer runtime preloaded; any report makes that process fail.  Only host
code runs: every call in tests/test_abi.py returns from host-side validation.
"""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc is needed to build the sanitized library")
def test_abi_tests_pass_under_host_sanitizers():
    sys.path.insert(0, ROOT)
    from paper_2106_12736_amd import build

    lib = build.build_host_sanitized(verbose=False)
    env = dict(os.environ)
    env["FDC_LIBRARY"] = lib
    env["LD_PRELOAD"] = build.asan_runtime()
    # leak checking is off: the interpreter and the HIP runtime keep allocations to exit
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "passed" in r.stdout
