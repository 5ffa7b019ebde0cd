"""The C ABI's host-side validation under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

api.hip is compiled with both sanitizers on its host code (the device code is
untouched), and tests/asan/abi_driver.c calls every entry point with arguments
host validation refuses, checking each status; the library's other
translation units come from the built libstepprune.so.  No call reaches the
device, so this runs without a GPU.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_13804_amd", "csrc")
LLVM = "/opt/rocm/llvm/bin"
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]


def test_abi_validation_under_sanitizers(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    clang = os.path.join(LLVM, "clang")
    if not (os.path.exists(hipcc) and os.path.exists(clang)):
        pytest.skip("hipcc or ROCm's clang is not available")
    from paper_2609_13804_amd import binding
    lib_dir = os.path.dirname(binding.LIB_PATH)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    api = tmp_path / "api_asan.o"
    drv = tmp_path / "abi_driver.o"
    exe = tmp_path / "abi_driver"
    run = lambda cmd: subprocess.run(cmd, check=True, capture_output=True, text=True, timeout=600)
    run([hipcc, "-O1", "-g", "-fPIC", "--offload-arch=gfx950", "-Xclang", "-target-feature",
         "-Xclang", "-packed-fp32-ops", *SANITIZE, *inc, "-c", os.path.join(CSRC, "api.hip"),
         "-o", str(api)])
    run([clang, "-std=c99", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-D__HIP_PLATFORM_AMD__", *inc, "-I", "/opt/rocm/include", "-c",
         os.path.join(ROOT, "tests", "asan", "abi_driver.c"), "-o", str(drv)])
    run([os.path.join(LLVM, "clang++"), "-fsanitize=address,undefined", str(drv), str(api),
         "-L", lib_dir, "-lstepprune", "-L", "/opt/rocm/lib", "-lamdhip64",
         "-lrocprofiler-sdk-roctx", f"-Wl,-rpath,{lib_dir}", "-Wl,-rpath,/opt/rocm/lib",
         "-o", str(exe)])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("ok: 0 failure(s)"), r.stdout
