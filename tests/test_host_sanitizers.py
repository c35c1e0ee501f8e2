"""The C ABI's host code under AddressSanitizer, LeakSanitizer and
UndefinedBehaviorSanitizer (CPU only): tests/host_san/abi_host_checks.cpp
drives argument validation, the error path of a context without a device,
calls on a NULL context and the temporal efficiency of Eq. 4 through a
host-sanitized build of the library; any sanitizer report fails the test."""
import os
import subprocess

import pytest

from tests.host_san import build as san_build


def _regular_objects_present():
    d = san_build.OBJS
    return os.path.isdir(d) and any(f.endswith(".o") for f in os.listdir(d))


@pytest.mark.timeout(600)
def test_abi_host_code_under_sanitizers(tmp_path):
    if not os.path.exists(san_build.HIPCC) or not os.path.exists(san_build.CLANG):
        pytest.skip("no ROCm toolchain")
    if not _regular_objects_present():
        from paper_1710_02368_amd import build as lib_build
        lib_build.build(verbose=False)
    exe = san_build.build(str(tmp_path))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "Sanitizer" not in out, out[-4000:]
    assert "0 failure(s)" in out, out[-4000:]
