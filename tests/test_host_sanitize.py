"""The C ABI under AddressSanitizer and UndefinedBehaviorSanitizer.

``tests/sanitize/host_abi_driver`` (built by ``build()``) holds tm_api.cpp
compiled with both sanitizers plus a driver that calls every entry point:
descriptor and argument checks, cache sizes, the planner's pair counts against
closed forms and brute force, and the size limits at INT32_MAX. Any sanitizer
report aborts the run. On a GPU it also drives the cache bookkeeping and every
launch through real device memory.
"""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "tests", "sanitize", "host_abi_driver")
ENV = dict(os.environ,
           ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
           LSAN_OPTIONS="suppressions=" + os.path.join(ROOT, "tests", "sanitize", "lsan.supp"))


def _run(*args):
    if not os.path.exists(DRIVER):
        pytest.skip("tests/sanitize/host_abi_driver is not built (run build())")
    res = subprocess.run([DRIVER, *args], capture_output=True, text=True, env=ENV, timeout=300)
    print(res.stdout[-3000:], res.stderr[-6000:])
    assert res.returncode == 0, res.stderr[-6000:]
    assert "all checks passed" in res.stdout


def test_host_abi_under_asan_and_ubsan():
    _run()


@pytest.mark.gpu
def test_device_paths_under_host_asan_and_ubsan():
    _run("--gpu")
