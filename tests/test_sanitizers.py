"""AddressSanitizer and UndefinedBehaviorSanitizer runs of the CPU oracle and of the library's host
code (no GPU needed).

* The oracle (oracle/oracle.c) is built with gcc and the sanitizers into a small driver
  (tests/sanitize/oracle_driver.c) that runs its forward and backward on problems reaching every
  indexing path: odd and one-row maps, K above the candidate count, both variants and storage
  types, one level, per-level K, given V levels, the position encoding and teacher forcing.
* The library's host code (every csrc source, sanitizers on the host side only; the device code is
  compiled as usual) is linked into a driver (tests/sanitize/abi_driver.cpp) that calls every
  entry point with arguments validation must reject, and the workspace queries with valid ones, so
  no call reaches a device.
Either build is skipped only when its compiler is missing."""
import glob
import os
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
CLANGXX = "/opt/rocm/llvm/bin/clang++"
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}"
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc missing")
def test_oracle_under_asan_and_ubsan():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "oracle_san")
        _run(["gcc", "-std=c11", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
              "-fno-omit-frame-pointer", "-Wall", "-Wextra", "-o", exe,
              os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"), "-lm"])
        r = _run([exe], env=ENV, timeout=300)
        assert "0 failures" in r.stdout


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANGXX)), reason="ROCm compilers missing")
def test_host_validation_under_asan_and_ubsan():
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2201_02767_amd", "csrc", "*.hip")))
    with tempfile.TemporaryDirectory() as d:
        def compile_one(src):
            obj = os.path.join(d, os.path.basename(src) + ".o")
            _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                  "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *SAN_HOST,
                  f"-I{os.path.join(ROOT, 'include')}", "-c", src, "-o", obj])
            return obj
        with ThreadPoolExecutor(max_workers=8) as ex:
            objs = list(ex.map(compile_one, srcs + [os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp")]))
        exe = os.path.join(d, "abi_san")
        _run([CLANGXX, "-fsanitize=address,undefined", "-o", exe, *objs, "-L/opt/rocm/lib", "-lamdhip64",
              "-Wl,-rpath,/opt/rocm/lib"])
        r = _run([exe], env=ENV, timeout=300)
        assert "0 failures" in r.stdout
