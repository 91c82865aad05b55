"""AddressSanitizer + UndefinedBehaviorSanitizer builds, run on the CPU.

- The oracle (plain C) with a driver that calls every one of its functions
  on small dense and CSR inputs, for both problem types and the four
  kernels, and its argument checks (tests/sanitize/oracle_driver.c).
- The library's host code (argument validation, status codes, error
  messages, dispatch) with a driver that feeds every entry point bad
  arguments and expects the right refusal (tests/sanitize/abi_driver.c).
  The device objects are the library's own, unchanged: the sanitizers
  instrument only the host side, and no call here reaches the GPU.

Any sanitizer report aborts the driver, and the test fails with its output.
"""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
PKG = os.path.join(ROOT, "paper_1706_05544_amd")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer", "-g", "-O1"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, "%s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr)
    return r


def test_oracle_under_asan_ubsan(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_asan")
    _run(["gcc", "-std=c11", "-fopenmp", "-Wall", "-Wextra"] + SAN +
         ["-I" + os.path.join(ROOT, "oracle"),
          os.path.join(HERE, "oracle_driver.c"),
          os.path.join(ROOT, "oracle", "svm_oracle.c"), "-lm", "-o", exe])
    r = _run([exe], env=ENV, timeout=300)
    assert "all checks passed" in r.stdout


def _device_objects():
    from paper_1706_05544_amd import build as b
    objs = [os.path.join(b.BUILD, s + ".o") for s in b.DEVICE_SOURCES]
    if not all(os.path.exists(o) for o in objs):
        b.build()
    return objs


def test_abi_validation_under_asan_ubsan(tmp_path):
    from paper_1706_05544_amd import build as b
    hipcc = b._hipcc()
    llvm = "/opt/rocm/llvm/bin"
    if not os.path.exists(os.path.join(llvm, "clang++")):
        pytest.skip("ROCm clang not found")
    # host code instrumented, device code as in the library; each sanitizer
    # flag applies to the host compilation only
    host_san = []
    for f in SAN[:3]:
        host_san += ["-Xarch_host", f]
    objs = []
    for src in b.HOST_SOURCES:
        o = str(tmp_path / (src + ".o"))
        _run([hipcc] + [c for c in b.COMMON if c != "-O3"] + ["-O1", "-g"] +
             host_san + ["-c", os.path.join(b.CSRC, src), "-o", o])
        objs.append(o)
    drv = str(tmp_path / "abi_driver.o")
    _run([os.path.join(llvm, "clang"), "-std=c11"] + SAN +
         ["-I" + b.INCLUDE, "-c", os.path.join(HERE, "abi_driver.c"),
          "-o", drv])
    exe = str(tmp_path / "abi_asan")
    _run([os.path.join(llvm, "clang++")] + SAN[:1] +
         ["-o", exe, drv] + objs + _device_objects() +
         ["-L/opt/rocm/lib", "-lamdhip64"] + b.LINK)
    r = _run([exe], env=ENV, timeout=300)
    assert "all checks passed" in r.stdout
