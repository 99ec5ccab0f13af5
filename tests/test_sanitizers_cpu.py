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
    drv, exe = str(tmp_path / "abi_driver.o"), str(tmp_path / "abi_san")
    rc, log = _run(["gcc", "-O1", "-g", "-std=c99", "-c", "-I", os.path.join(ROOT, "include"),
                    os.path.join(SAN, "abi_driver.c"), "-o", drv])
    assert rc == 0, log
    # host-only sanitizers on the library: each -fsanitize= right after -Xarch_host
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
    # the three translation units compile concurrently (device code unoptimised:
    # nothing here launches a kernel)
    objs, procs = [], []
    for src in ("sched_kernels.hip", "sched_wide.hip", "sched_group.hip", "opt_kernels.hip"):
        obj = str(tmp_path / (src + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen([hipcc, "--offload-arch=gfx950", "-Xarch_device", "-O0", "-O1", "-g",
                                       "-std=c++17", *san, "-I", os.path.join(ROOT, "include"), "-c",
                                       os.path.join(ROOT, "paper_2508_14544_amd", "csrc", src), "-o", obj],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
    for pr in procs:
        log = pr.communicate(timeout=900)[0]
        assert pr.returncode == 0, log
    rc, log = _run([hipcc, "--offload-arch=gfx950", *san, *objs, drv, "-o", exe], timeout=300)
    assert rc == 0, log
    rc, log = _run([exe], env=ENV, timeout=120)
    assert rc == 0 and "ERROR: AddressSanitizer" not in log and "runtime error" not in log, log
