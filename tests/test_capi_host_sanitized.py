"""The host C-ABI checks of test_capi_host.py against a build of the C ABI
with AddressSanitizer and UndefinedBehaviorSanitizer on its host code (kernel
objects unchanged, no GPU call is made).  Any sanitizer report fails the run."""
import shutil

import pytest

import hostsan_build


def test_capi_host_checks_under_asan_and_ubsan():
    runtime = hostsan_build.asan_runtime()
    if runtime is None or shutil.which("python3") is None:
        pytest.skip("no ASan runtime in the ROCm toolchain")
    lib = hostsan_build.build()
    r = hostsan_build.run_host_tests(lib, runtime)
    out = r.stdout
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in out and " failed" not in out, out[-3000:]
