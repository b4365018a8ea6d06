"""The C-ABI checks under AddressSanitizer and UndefinedBehaviorSanitizer.

The library's host code (argument validation, shape and overflow checks,
workspace planning, option parsing, status strings) is rebuilt with the
sanitizers on the host side only and the ABI and binding tests are run
against it in a child process, with the sanitizer runtime preloaded and any
report fatal.  No kernel is launched: every call fails validation first."""

import os
import subprocess
import sys

import pytest

from paper_1709_02755_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def sanitized_lib():
    try:
        return build.build_sanitized()
    except RuntimeError as e:  # no ROCm toolchain at all
        pytest.skip(f"cannot build the sanitized library: {e}")


def test_abi_checks_are_clean_under_asan_and_ubsan(sanitized_lib):
    env = dict(os.environ)
    env.update(LD_PRELOAD=build.sanitizer_runtime(), SRU_LIBRARY=sanitized_lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    probe = ("import sys; sys.path.insert(0, %r); from paper_1709_02755_amd import sru; "
             "sru.lib(); maps = open('/proc/self/maps').read(); "
             "assert 'libclang_rt.asan' in maps and %r in maps; print('sanitized')"
             % (ROOT, os.path.basename(sanitized_lib)))
    r = subprocess.run([sys.executable, "-c", probe], env=env, capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0 and "sanitized" in r.stdout, r.stderr[-2000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py"),
                        os.path.join(ROOT, "tests", "test_binding_host.py")],
                       env=env, capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr
    assert "runtime error:" not in r.stderr
