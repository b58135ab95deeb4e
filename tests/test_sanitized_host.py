"""The host side of the library (argument validation, workspace planning,
launch sequencing, the C ABI) under AddressSanitizer and
UndefinedBehaviorSanitizer: the host ABI tests run clean against a copy of the
library whose host code is instrumented (device code unchanged; no GPU needed)."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.slow
def test_host_abi_tests_clean_under_asan_ubsan():
    from paper_2608_09703_amd import build_lib
    lib = build_lib.build(sanitize=True)
    env = dict(os.environ)
    env.update({"LD_PRELOAD": build_lib.sanitizer_runtime(), "MLS_LIBRARY": lib,
                "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"})
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_host.py")], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-3000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-3000:]
    # the instrumented copy was the one loaded
    probe = subprocess.run([sys.executable, "-c", "from paper_2608_09703_amd import binding as B; "
                            "B.lib(); print(any('libmls_san.so' in l for l in open('/proc/self/maps')))"],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert probe.stdout.strip().endswith("True"), probe.stdout + probe.stderr
