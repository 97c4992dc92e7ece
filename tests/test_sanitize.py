"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The host side of every entry point (argument validation, launch plans,
workspace sizes and layouts) is built with -fsanitize=address,undefined and
no device code, and tests/test_abi.py runs against it in a child process that
preloads the ASan runtime.  Any invalid access or undefined behaviour aborts
the child, which fails this test.  CPU only: nothing in that build can
launch a kernel.
"""

import os
import subprocess
import sys

from tests._util import ROOT


def test_abi_validation_under_asan_and_ubsan():
    from paper_2607_14107_amd import build
    lib = build.build_sanitized()
    rt = build.asan_runtime()
    assert os.path.exists(rt), rt
    env = dict(os.environ)
    env.update(POLESTAR_LIB=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    report = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, report
    assert "runtime error" not in report and "AddressSanitizer" not in report, report
    assert " passed" in r.stdout, report
