"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two programs are built in a temporary directory and run:

* the library's host code -- the C ABI entry points, argument and plan
  checks, the plan enumeration and time model (cnn_api.cpp, cnn_select.cpp)
  and the host side of every kernel source (variant tables, launch
  wrappers) -- with the sanitizers on the host side only; the device code
  is compiled as in the product build and never runs (no GPU is used:
  every call the driver makes returns before any HIP call);
* the fp64 oracle (conv_oracle.c), built with gcc.

UBSan is built non-recovering, so the first report aborts the program and
fails the test.
"""
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2105_13480_amd import build as libbuild  # noqa: E402

HERE = os.path.join(ROOT, "tests", "sanitize")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")

# every sanitizer flag applies to host code only
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined"]


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout[-4000:]}\n{res.stderr[-4000:]}"
    return res


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_library_host_code_sanitized():
    common = ["--offload-arch=" + libbuild.ARCH, "-O1", "-g", "-fno-omit-frame-pointer",
              "-std=c++17", "-fPIC", "-I", os.path.join(ROOT, "include")] + HOST_SAN
    device = ["-Xarch_device", "-O3", "-Xarch_device", "-g0"] + libbuild.HIP_ONLY
    with tempfile.TemporaryDirectory() as tmp:
        procs, objs = [], []
        for src in libbuild.SOURCES:
            obj = os.path.join(tmp, src + ".o")
            cmd = [HIPCC] + common
            if src.endswith(".hip"):
                cmd += ["-x", "hip"] + device
            cmd += ["-c", os.path.join(libbuild.CSRC, src), "-o", obj]
            procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                stderr=subprocess.PIPE, text=True)))
            objs.append(obj)
        for cmd, p in procs:
            out, err = p.communicate()
            assert p.returncode == 0, f"{' '.join(cmd)}\n{err[-4000:]}"
        drv_obj = os.path.join(tmp, "driver.o")
        _run([HIPCC] + common + ["-x", "c++", "-c", os.path.join(HERE, "lib_host_driver.c"),
                                 "-o", drv_obj])
        exe = os.path.join(tmp, "lib_host_driver")
        _run([HIPCC] + HOST_SAN[:4] + objs + [drv_obj, "-o", exe])
        res = _run([exe], env=ENV, timeout=600)
        assert "ok" in res.stdout and "runtime error" not in res.stderr, res.stderr[-4000:]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_sanitized():
    with tempfile.TemporaryDirectory() as tmp:
        exe = os.path.join(tmp, "oracle_driver")
        _run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
              "-fno-sanitize-recover=undefined", "-fopenmp", "-o", exe,
              os.path.join(HERE, "oracle_driver.c"), os.path.join(ROOT, "oracle", "conv_oracle.c"),
              "-lm"])
        res = _run([exe], env=ENV, timeout=300)
        assert "ok" in res.stdout and "runtime error" not in res.stderr, res.stderr[-4000:]
