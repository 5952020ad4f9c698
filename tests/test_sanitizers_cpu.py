"""AddressSanitizer / UndefinedBehaviorSanitizer builds of host code, run on
the CPU (no GPU needed):

* the fp64 oracle (oracle/kvr_ref.c) with a driver that runs every entry
  point on tiny shapes and thread counts, with NaN canaries around the cache
  rows it must not touch (tests/sanitize/oracle_driver.c);
* libkvr's host code (argument validation, split planning, workspace
  layouts, artifact headers: csrc/kvr_api.hip and csrc/artifact.hip) with a
  driver whose kernel launchers are stubs: fixed rejection cases, every
  corrupted header byte, and a deterministic fuzz of descriptors, lengths and
  reader tables (tests/sanitize/host_driver.cpp).

Sanitizers are applied to host code only; device code is not instrumented.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2606_13361_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

ENV = dict(os.environ,
           ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _check(proc):
    out = proc.stdout.decode(errors="replace") + proc.stderr.decode(errors="replace")
    assert proc.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    return out


def test_oracle_under_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_driver")
    subprocess.run([gcc, "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-pthread", os.path.join(ROOT, "oracle", "kvr_ref.c"),
                    os.path.join(SAN, "oracle_driver.c"), "-lm", "-o", exe], check=True)
    out = _check(subprocess.run([exe], env=ENV, capture_output=True, timeout=600))
    assert "all checks passed" in out


def test_library_host_code_under_sanitizers(tmp_path):
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    clang = os.path.join(ROCM, "llvm", "bin", "clang++")
    if not (os.path.exists(hipcc) and os.path.exists(clang)):
        pytest.skip("ROCm compilers not available")
    # host-side instrumentation only: every sanitizer flag goes to the host pass
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    objs = []
    for src in (os.path.join(CSRC, "kvr_api.hip"), os.path.join(CSRC, "artifact.hip"),
                os.path.join(SAN, "host_driver.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        subprocess.run([hipcc, "-x", "hip", "-c", "-fPIC", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + host_san +
                       ["-I" + INCLUDE, "-I" + CSRC, src, "-o", obj], check=True, capture_output=True)
        objs.append(obj)
    exe = str(tmp_path / "host_driver")
    subprocess.run([clang, "-fsanitize=address,undefined"] + objs +
                   ["-L" + os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"),
                    "-o", exe], check=True)
    out = _check(subprocess.run([exe], env=ENV, capture_output=True, timeout=600))
    assert "all checks passed" in out
