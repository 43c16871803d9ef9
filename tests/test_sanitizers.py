"""CPU runs under the address and undefined-behaviour sanitizers:

* the oracle (oracle/qnn_oracle.c) with a driver that calls every entry
  point on small seeded inputs (oracle/sanitize_check.c), built with gcc;
* the library's host code (csrc/qnn_api.cpp: argument validation, the
  fixed-point multiplier, the kernel-choice file parser, NULL handling),
  built with the sanitizers on its host side only (the device code is
  unchanged) and linked with the other library objects and a driver that
  reaches no device work (tests/sanitize/abi_check.cpp).

A sanitizer report or a nonzero exit fails the test."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="2")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, (cmd if isinstance(cmd, str) else " ".join(cmd)) + "\n" + (r.stdout + r.stderr)[-4000:]
    return r


@pytest.mark.skipif(not shutil.which("gcc"), reason="gcc not available")
def test_oracle_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_san"
    _run(["gcc", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
          "-fopenmp", "-std=c11", "-Wall", "-Wextra", os.path.join(ROOT, "oracle", "sanitize_check.c"),
          os.path.join(ROOT, "oracle", "qnn_oracle.c"), "-o", str(exe), "-lm"])
    r = _run([str(exe)], env=SAN_ENV, timeout=300)
    assert "oracle sanitizer run done" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-2000:]


def _library_objects():
    objs = sorted(glob.glob(os.path.join(ROOT, "paper_2006_10226_amd", "_build", "*.o")))
    return [o for o in objs if os.path.basename(o) != "qnn_api.o"
            and os.path.basename(o)[:-2] + ".hip" in os.listdir(os.path.join(ROOT, "paper_2006_10226_amd", "csrc"))]


@pytest.mark.skipif(not os.path.exists(HIPCC) or not os.path.exists(CLANG), reason="ROCm compilers not available")
def test_library_host_code_under_sanitizers(tmp_path):
    objs = _library_objects()
    if not objs:
        pytest.skip("library objects not built (run the build first)")
    csrc = os.path.join(ROOT, "paper_2006_10226_amd", "csrc")
    api = tmp_path / "qnn_api_san.o"
    # sanitizers on the host side only: each -fsanitize= follows -Xarch_host
    _run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
          "-I" + os.path.join(ROOT, "include"), "-I" + csrc,
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
          "-Xarch_host", "-fno-omit-frame-pointer",
          "-c", os.path.join(csrc, "qnn_api.cpp"), "-o", str(api)])
    drv = tmp_path / "abi_check.o"
    _run([CLANG, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
          "-I" + os.path.join(ROOT, "include"), "-c", os.path.join(ROOT, "tests", "sanitize", "abi_check.cpp"),
          "-o", str(drv)])
    exe = tmp_path / "abi_san"
    _run([CLANG, "-fsanitize=address,undefined", "-o", str(exe), str(drv), str(api), *objs, "-L/opt/rocm/lib",
          "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    r = _run([str(exe), str(tmp_path / "choices.txt")], env=SAN_ENV, timeout=300)
    assert "abi sanitizer run done" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-2000:]
