"""Host code of the library under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds the sanitized copy of libsphinx.so (host code instrumented, device code
as usual) and runs the CPU tests of the C ABI against it in a subprocess with
the sanitizer runtime preloaded: every argument check and error path of every
entry point, the request tables, the step, cache and grid planners and the
adaptive start-step computation.  Any sanitizer report fails the test.  No GPU
is touched (the ABI tests make no compute call without one).
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_abi_under_asan_and_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2511_18672_amd import build as B

    lib = B.build_sanitized()
    env = dict(os.environ)
    env.update(SPHINX_LIBRARY=lib, LD_PRELOAD=B.sanitizer_runtime(),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py"), os.path.join(ROOT, "tests", "test_adaptive_start.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    print(out[-3000:])
    assert "runtime error" not in out and "AddressSanitizer" not in out
    assert r.returncode == 0
    assert " passed" in out
