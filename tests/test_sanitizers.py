"""Host code under the address and undefined-behaviour sanitizers (CPU).

The fp64 oracle is compiled with gcc into a driver that runs it through
every option (tests/sanitize/oracle_driver.c); the library's host side is
compiled with hipcc, the sanitizers on its host pass only, and a clang-built
C driver calls every entry point that enqueues nothing over valid, extreme
and invalid configurations (tests/sanitize/abi_driver.c).  Either run must
finish cleanly: exit status 0 and no sanitizer report.  GPU code is not
instrumented (device sanitizers are not available here)."""
import os
import shutil
import subprocess

import pytest

from paper_2508_01744_amd import _build

HERE = os.path.dirname(os.path.abspath(__file__))
SAN = os.path.join(HERE, "sanitize")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.environ.get("HIPCC", os.path.join(ROCM, "bin", "hipcc"))
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
REPORT_MARKS = ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer")


def _run_clean(exe, env_extra=None):
    env = dict(os.environ, UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", **(env_extra or {}))
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert not any(m in out for m in REPORT_MARKS), out[-4000:]
    return out


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.run(["gcc", "-std=c99", "-O1", "-g", "-Wall", "-Wno-unknown-pragmas",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-fno-omit-frame-pointer", os.path.join(SAN, "oracle_driver.c"), "-o", exe, "-lm"],
                   check=True)
    out = _run_clean(exe, {"ASAN_OPTIONS": "detect_leaks=1"})
    assert "0 failures" in out


@pytest.mark.skipif(not os.path.exists(HIPCC) or not os.path.exists(CLANG), reason="hipcc or clang not found")
def test_library_host_side_under_sanitizers(tmp_path):
    lib = str(tmp_path / "libagft_san.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC", "-shared", "-w",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-I", _build.INCLUDE, *_build.SOURCES, "-o", lib]
    subprocess.run(cmd, check=True)
    exe = str(tmp_path / "abi_driver")
    subprocess.run([CLANG, "-std=c11", "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                    "-D__HIP_PLATFORM_AMD__", "-I", _build.INCLUDE, "-I", os.path.join(ROCM, "include"),
                    os.path.join(SAN, "abi_driver.c"), lib, "-Wl,-rpath," + str(tmp_path), "-o", exe],
                   check=True)
    # the HIP runtime the library links is not instrumented; its allocations
    # at load time are not this code's leaks
    out = _run_clean(exe, {"ASAN_OPTIONS": "detect_leaks=0"})
    assert "0 failures" in out
