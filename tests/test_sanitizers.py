"""CPU sanitizer targets: the oracle, and the library's host-side paths that
run before any device call (argument validation, the plan query, status
strings, the profiling hook), each built with AddressSanitizer and
UndefinedBehaviorSanitizer and driven by a small program under
tests/sanitize/.  No GPU is needed; any sanitizer report fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
ENV = dict(os.environ, ASAN_OPTIONS="abort_on_error=1:detect_leaks=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


def _run(cmd, env=None, timeout=600):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    return r.returncode, r.stdout + r.stderr


def _clean(log):
    return "AddressSanitizer" not in log and "runtime error" not in log and "LeakSanitizer" not in log


def test_oracle_under_asan_and_ubsan(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_sanitized")
    rc, log = _run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-std=c11",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "oracle", "exemcl_oracle.c"), os.path.join(HERE, "oracle_driver.c"),
                    "-o", exe, "-lm"])
    assert rc == 0, log
    rc, log = _run([exe], env=ENV)
    assert rc == 0 and _clean(log) and "oracle checks passed" in log, log


def test_host_validation_under_asan_and_ubsan(tmp_path):
    from paper_2101_08763_amd import build as B
    if not os.path.exists(B.HIPCC):
        pytest.skip("hipcc not available")
    os.makedirs(B.OBJDIR, exist_ok=True)
    kernel_objs = []
    for src in B.SOURCES:
        if src == "host.cpp":
            continue
        obj = os.path.join(B.OBJDIR, os.path.splitext(src)[0] + ".o")
        if not os.path.exists(obj):
            B._compile(src, False)
        kernel_objs.append(obj)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in B.FLAGS if f != "-fvisibility=hidden"]
    host_obj = str(tmp_path / "host_sanitized.o")
    rc, log = _run([B.HIPCC, *flags, *san, "-g", "-x", "hip", "-c", os.path.join(B.CSRC, "host.cpp"),
                    "-o", host_obj])
    assert rc == 0, log
    drv_obj = str(tmp_path / "host_driver.o")
    rc, log = _run([B.HIPCC, "-O1", "-g", "-std=c++17", f"-I{B.INCLUDE}", *san, "-c",
                    os.path.join(HERE, "host_driver.cpp"), "-o", drv_obj])
    assert rc == 0, log
    exe = str(tmp_path / "host_sanitized")
    rc, log = _run([B.HIPCC, f"--offload-arch={B.ARCH}", *san, host_obj, drv_obj, *kernel_objs, "-o", exe])
    assert rc == 0, log
    # the HIP runtime keeps allocations for the life of the process
    env = dict(ENV, ASAN_OPTIONS="abort_on_error=1:detect_leaks=0")
    rc, log = _run([exe], env=env)
    assert rc == 0 and _clean(log) and "host checks passed" in log, log
