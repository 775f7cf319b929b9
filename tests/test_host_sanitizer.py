"""The host logic (planner, argument checks, C ABI, exchange ring, streaming
copy entry point) built with the host compiler's address and
undefined-behaviour sanitizers, and the host ABI tests run against that build
in a child process with the sanitizer runtime preloaded: any out-of-bounds
access, use after free or undefined behaviour on those paths ends the run
with a report."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from paper_2607_23089_amd import build as B  # noqa: E402


@pytest.fixture(scope="module")
def check_lib(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("host_check") / "librowsm_check.so")
    return B.build_host_check(out, os.path.join(ROOT, "tests", "host_check",
                                                "launcher_stubs.hip"))


def test_host_abi_tests_under_sanitizers(check_lib):
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": B.sanitizer_runtime(),
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "ROWSM_LIB": check_lib,
    })
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi_host.py")],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = res.stdout + res.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert res.returncode == 0, out[-4000:]
    assert " passed" in out
