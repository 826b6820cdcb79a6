"""The C ABI's host layer under AddressSanitizer and UndefinedBehaviorSanitizer.

The library is rebuilt with both sanitizers on its host code (the device code
is compiled as usual and never runs), and tests/abi_sanitize.c drives every
entry point's argument validation (configurations, cache views, region
tables, calls on a NULL handle) and the host-only fit of md_calib_fit.  All
of it returns before the HIP runtime is used, so no GPU is needed; the
sanitizers stop the run at the first invalid access or undefined operation.
"""
import os
import subprocess

import pytest

from paper_2607_10582_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
CSRC = os.path.join(ROOT, "paper_2607_10582_amd", "csrc")
CLANG = "/opt/rocm/lib/llvm/bin/clang"


def test_host_layer_under_sanitizers(tmp_path):
    if not os.path.exists(CLANG):
        pytest.fail(f"{CLANG} is missing (ROCm's clang builds the sanitized driver)")
    lib = tmp_path / "libmemdecay_san.so"
    srcs = [os.path.join(CSRC, s) for s in build.SOURCES]
    # sanitizers on the host code only: each -fsanitize= follows -Xarch_host
    cmd = [build.hipcc(), "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", INCLUDE, *srcs, "-o", str(lib)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    exe = tmp_path / "abi_sanitize"
    drv = [CLANG, "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-g", "-I", INCLUDE,
           os.path.join(ROOT, "tests", "abi_sanitize.c"), str(lib), f"-Wl,-rpath,{tmp_path}", "-lm", "-o", str(exe)]
    r = subprocess.run(drv, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "passed under the sanitizers" in r.stdout
