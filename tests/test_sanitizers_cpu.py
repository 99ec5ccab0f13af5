"""Host sanitizer builds (CPU only): the C oracle under AddressSanitizer and
UndefinedBehaviorSanitizer over random instances, and the library's host-side
argument checks under host AddressSanitizer and UndefinedBehaviorSanitizer
(the device code is not sanitized; no call here reaches the GPU)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    return r.returncode, r.stdout + r.stderr


def test_oracle_under_asan_ubsan(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_san")
    rc, log = _run(["gcc", "-O1", "-g", "-std=c99", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "oracle"),
                    os.path.join(ROOT, "oracle", "sched_oracle.c"), os.path.join(SAN, "oracle_driver.c"), "-o", exe])
    assert rc == 0, log
    rc, log = _run([exe, "3000"], env=ENV, timeout=300)
    assert rc == 0 and "ERROR" not in log and "runtime error" not in log, log


def test_library_host_checks_under_asan_ubsan(tmp_path):
    hipcc = "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not shutil.which("gcc"):
        pytest.skip("hipcc or gcc not found")
    drv, lib, exe = str(tmp_path / "abi_driver.o"), str(tmp_path / "sk.o"), str(tmp_path / "abi_san")
    rc, log = _run(["gcc", "-O1", "-g", "-std=c99", "-c", "-I", os.path.join(ROOT, "include"),
                    os.path.join(SAN, "abi_driver.c"), "-o", drv])
    assert rc == 0, log
    # host-only sanitizers on the library: each -fsanitize= right after -Xarch_host
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
    rc, log = _run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", *san, "-Xclang", "-target-feature",
                    "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-c",
                    os.path.join(ROOT, "paper_2508_14544_amd", "csrc", "sched_kernels.hip"), "-o", lib], timeout=900)
    assert rc == 0, log
    rc, log = _run([hipcc, "--offload-arch=gfx950", *san, lib, drv, "-o", exe], timeout=300)
    assert rc == 0, log
    rc, log = _run([exe], env=ENV, timeout=120)
    assert rc == 0 and "ERROR: AddressSanitizer" not in log and "runtime error" not in log, log
