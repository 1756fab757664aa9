"""Builds the host-sanitised variant of librlx.so for the CPU tests: capi.hip
(the C ABI: argument validation, handle and workspace management, graph
cache) compiled with AddressSanitizer and UndefinedBehaviorSanitizer on its
host code only, linked with the regular kernel objects of the normal build.
Device code is not instrumented.  The library needs the ASan runtime loaded
first (LD_PRELOAD of ``asan_runtime()``), so the tests run in a child process.
"""
import glob
import os
import subprocess

from paper_2609_37916_amd import _build

SAN_LIB = os.path.join(_build.BUILD_DIR, "librlx_hostsan.so")


def asan_runtime():
    """The clang ASan shared runtime of the ROCm toolchain, or None."""
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so") +
                  glob.glob("/opt/rocm/llvm/lib/clang/*/lib/x86_64-unknown-linux-gnu/libclang_rt.asan.so"))
    return hits[-1] if hits else None


def build() -> str:
    cc = _build.hipcc()
    others = [s for s in _build.SOURCES if s != "capi.hip"]
    objs = [os.path.join(_build.BUILD_DIR, s.replace(".hip", ".o")) for s in others]
    if not all(os.path.exists(o) for o in objs):
        _build.build_library()
    san_obj = os.path.join(_build.BUILD_DIR, "capi_hostsan.o")
    base = [f"--offload-arch={_build.ARCH}", "-O1", "-g", "-std=c++17", "-fPIC", "-fno-omit-frame-pointer",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", os.path.join(_build.ROOT, "include")]
    # every sanitiser flag applies to the host pass only
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined"]
    _build._run([cc, *base, *san, "-c", os.path.join(_build.CSRC, "capi.hip"), "-o", san_obj], False)
    _build._run([cc, f"--offload-arch={_build.ARCH}", "-shared", "-fPIC", *san, "-shared-libasan", san_obj, *objs,
                 "-o", SAN_LIB], False)
    return SAN_LIB


def run_host_tests(lib_path, runtime):
    """Runs tests/test_capi_host.py against `lib_path` in a child process."""
    root = _build.ROOT
    env = dict(os.environ, LD_PRELOAD=runtime, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", PYTHONPATH=root)
    code = ("import sys, pytest, paper_2609_37916_amd as rlx; rlx.LIB_PATH = sys.argv[1]; "
            "sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', 'tests/test_capi_host.py']))")
    return subprocess.run(["python3", "-c", code, lib_path], cwd=root, env=env, stdout=subprocess.PIPE,
                          stderr=subprocess.STDOUT, text=True, timeout=600)
