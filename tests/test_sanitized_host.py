"""The host code of the library under AddressSanitizer + UndefinedBehaviorSanitizer
and under ThreadSanitizer (CPU only).

__graft_entry__.build() also builds libpointid_asan.so and libpointid_tsan.so:
the same sources with the host code instrumented (every -fsanitize= flag
passed with -Xarch_host; the device code is untouched).  Each test runs
tests/test_abi_host.py -- argument validation of every entry point, the batcher
and server set-up paths, and the socket client's framing against a stub server
thread -- in a child process that loads the sanitized build (POINTID_LIB) with
its runtime preloaded, and fails on any sanitizer report.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2009_04509_amd import build as B  # noqa: E402  (build helpers only, no GPU)

OPTIONS = {
    "address": ("ASAN_OPTIONS", "detect_leaks=0:halt_on_error=1:abort_on_error=0",
                ("ERROR: AddressSanitizer", "runtime error:")),
    "thread": ("TSAN_OPTIONS", "halt_on_error=1:report_signal_unsafe=0",
               ("WARNING: ThreadSanitizer", "ERROR: ThreadSanitizer")),
}


@pytest.mark.parametrize("sanitize", ["address", "thread"])
def test_host_abi_under_sanitizer(sanitize):
    lib = B.library_path(sanitize)
    rt = B.sanitizer_runtime(sanitize)
    if not os.path.exists(lib):
        pytest.skip(f"{os.path.basename(lib)} is not built (__graft_entry__.build() builds it)")
    if rt is None:
        pytest.skip(f"no clang {sanitize} runtime found under the ROCm LLVM")
    var, opts, marks = OPTIONS[sanitize]
    env = dict(os.environ, POINTID_LIB=lib, LD_PRELOAD=rt, UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env[var] = opts
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "passed" in out and not any(m in out for m in marks), out[-4000:]
    # the child really ran on the sanitized build
    probe = subprocess.run([sys.executable, "-c", "from paper_2009_04509_amd import binding as b; "
                            "print(b.LIB_PATH)"], cwd=ROOT, env=env, capture_output=True, text=True,
                           timeout=300)
    assert probe.returncode == 0 and probe.stdout.strip() == lib, probe.stdout + probe.stderr
