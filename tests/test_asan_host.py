"""The C ABI's host code (pool allocator, validation, work lists, table
checks, trace layouts) under AddressSanitizer and UndefinedBehaviorSanitizer.

``api.cpp`` is compiled for the host only, with the sanitizers on the host
side, and linked with launchers that launch nothing (tests/asan); the
driver ``abi_host_check.cpp`` exercises every host path with randomised
inputs.  No GPU is used.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
CLANGXX = os.path.join(ROCM, "llvm", "bin", "clang++")


def _run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


def test_host_abi_under_asan_and_ubsan(tmp_path):
    if not (os.path.exists(HIPCC) and os.path.exists(CLANGXX)):
        pytest.skip("ROCm compilers not found")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2510_14126_amd", "csrc")]
    host_hip = [HIPCC, "-x", "hip", "--offload-host-only", "--offload-arch=gfx950", "-O1", "-g",
                "-std=c++17", "-fno-omit-frame-pointer",
                "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all", *inc]
    _run(host_hip + ["-c", os.path.join(ROOT, "paper_2510_14126_amd", "csrc", "api.cpp"), "-o", "api.o"],
         tmp_path)
    _run(host_hip + ["-c", os.path.join(HERE, "asan", "launch_stubs.cpp"), "-o", "stubs.o"], tmp_path)
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    _run([CLANGXX, "-O1", "-g", "-std=c++17", *san, *inc, "-c",
          os.path.join(HERE, "asan", "abi_host_check.cpp"), "-o", "check.o"], tmp_path)
    lib = os.path.join(ROCM, "lib")
    _run([CLANGXX, *san, "api.o", "stubs.o", "check.o", "-L", lib, "-lamdhip64",
          f"-Wl,-rpath,{lib}", "-o", "abi_check"], tmp_path)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(tmp_path / "abi_check")], capture_output=True, text=True, env=env,
                       timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host ABI checks passed" in r.stdout
    assert "Sanitizer" not in r.stderr, r.stderr
