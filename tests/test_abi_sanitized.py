"""The C ABI's argument checks under AddressSanitizer and
UndefinedBehaviorSanitizer (host code; no GPU).

The library is rebuilt with host-side instrumentation when its sources
change, and tests/test_abi.py runs against it in a child process with the
sanitizer runtime preloaded: every validation path must pass without a
sanitizer report.
"""

import os
import subprocess
import sys

from paper_2211_17111_amd import build as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_validation_under_sanitizers():
    lib = b.build_sanitized()
    runtime = b.sanitizer_runtime()
    assert os.path.exists(runtime), runtime
    env = dict(os.environ)
    env.update(LD_PRELOAD=runtime, BEVPOOL_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi.py")],
                         cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                         timeout=900)
    out = res.stdout
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert res.returncode == 0, out[-4000:]
    assert " passed" in out
