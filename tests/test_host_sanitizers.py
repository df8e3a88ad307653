"""The C ABI's host side (argument checks, workspace layouts, split records,
the feature-cache sampler) under AddressSanitizer and UndefinedBehaviorSanitizer:
the library's host code is rebuilt instrumented (build_sanitized.py, no device
code) and tests/test_abi.py runs against it in a child python with the ASan
runtime preloaded.  Any sanitizer report aborts the child and fails the test."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(shutil.which("hipcc") is None and
                                not os.path.exists("/opt/rocm/bin/hipcc"),
                                reason="hipcc not available")


def test_abi_checks_clean_under_asan_and_ubsan():
    from paper_2606_00395_amd import build_sanitized as S
    lib = S.build()
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": S.runtime_preload(),
        "PR2_LIBRARY": lib,
        # python itself is not instrumented: its allocations are not leak-checked
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "HIP_VISIBLE_DEVICES": "",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"),
                        "-q", "-x", "-s", "-p", "no:cacheprovider"], cwd=ROOT, env=env,
                       stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
    lines = r.stdout.splitlines()
    report = [i for i, l in enumerate(lines) if "runtime error" in l or "ERROR: AddressSanitizer" in l]
    tail = "\n".join(lines[report[0]:report[0] + 12] if report else lines[-30:])
    assert r.returncode == 0, tail
    assert "passed" in tail and "ERROR: AddressSanitizer" not in r.stdout
    assert "runtime error" not in r.stdout, tail
