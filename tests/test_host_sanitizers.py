"""The host side of the C interface under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU.

pda_host.cpp (argument validation, launch plan, workspace layout) is built by
the host C++ compiler, instrumented, into a shared library with stand-ins for
the kernel launchers (tests/sanitize/kernel_stubs.cpp); the host-only ABI
tests then run against it through the binding's PDA_LIBRARY switch, with the
sanitizer runtime preloaded into the test process. Any report (a bad access,
an overflow, undefined behaviour) fails the run.
"""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_20863_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
# ABI tests that need more than the host code: the one-runtime check looks at
# which HIP runtime the process maps (the instrumented build links ROCm's own).
SKIP = "not one_hip_runtime"


def _gxx():
    return shutil.which("g++")


@pytest.mark.skipif(_gxx() is None or not os.path.exists(os.path.join(ROCM, "include", "hip")),
                    reason="needs g++ and the ROCm headers")
def test_host_code_under_asan_and_ubsan(tmp_path):
    gxx = _gxx()
    lib = str(tmp_path / "libpda_host_sanitized.so")
    build = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fPIC", "-shared",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
             "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
             "-I", CSRC, os.path.join(CSRC, "pda_host.cpp"), os.path.join(ROOT, "tests", "sanitize", "kernel_stubs.cpp"),
             "-L", os.path.join(ROCM, "lib"), f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-lamdhip64", "-o", lib]
    res = subprocess.run(build, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    asan_rt = subprocess.run([gxx, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    ubsan_rt = subprocess.run([gxx, "-print-file-name=libubsan.so"], capture_output=True, text=True).stdout.strip()
    env = dict(os.environ)
    env.update(PDA_LIBRARY=lib, LD_PRELOAD=" ".join(p for p in (asan_rt, ubsan_rt) if os.path.isabs(p)),
               # Python's own allocations are not this library's leaks
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi.py"), "-k", SKIP],
                         capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-6000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-6000:]
    assert " passed" in out
