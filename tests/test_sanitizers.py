"""AddressSanitizer and UndefinedBehaviorSanitizer runs on the CPU.

* The C oracle, built with gcc -fsanitize=address,undefined together with
  tests/sanitize/oracle_driver.c, runs every oracle entry point on small
  inputs (leak checking on).
* libpdec's host logic: the library's sources are compiled with the
  sanitizers on the host side only (-Xarch_host; the gfx950 device code is
  built as usual and never runs here) and linked with
  tests/sanitize/host_driver.c, which sweeps the planner, the length check
  and the argument checks of every launching entry point (all refused before
  any launch).

Either driver exits non-zero on a failed check, and the sanitizers abort on
the first report (-fno-sanitize-recover)."""
import concurrent.futures
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
HIPCC = "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"
SAN_ENV = dict(os.environ, ASAN_OPTIONS="abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout[-3000:] + r.stderr[-3000:]
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-O1", "-g", "-fopenmp", "-std=c11", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
          "-fno-omit-frame-pointer", "-Wall", "-Wextra", "-Werror", os.path.join(HERE, "oracle_driver.c"), "-o", exe,
          "-lm"])
    r = _run([exe], env=dict(SAN_ENV, ASAN_OPTIONS="abort_on_error=1:detect_leaks=1", OMP_NUM_THREADS="2"),
             timeout=300)
    assert "ok" in r.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_host_library_under_asan_and_ubsan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2607_02963_amd", "csrc")
    inc = os.path.join(ROOT, "include")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    srcs = sorted(f for f in os.listdir(csrc) if f.endswith(".hip"))

    def compile_one(f):
        obj = str(tmp_path / (f + ".o"))
        _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Xclang", "-target-feature",
              "-Xclang", "-packed-fp32-ops", "-Wno-unused-command-line-argument", *san, "-I", inc, "-I", csrc, "-c",
              os.path.join(csrc, f), "-o", obj])
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, srcs))
    drv = str(tmp_path / "host_driver.o")
    _run([CLANG, "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
          "-fno-omit-frame-pointer", "-Wall", "-Werror", "-I", inc, "-c", os.path.join(HERE, "host_driver.c"), "-o",
          drv])
    exe = str(tmp_path / "host_driver")
    _run([HIPCC, "--offload-arch=gfx950", *san, drv, *objs, "-o", exe])
    # the HIP runtime's own allocations are not this library's: leaks are not checked here
    r = _run([exe], env=dict(SAN_ENV, ASAN_OPTIONS="abort_on_error=1:detect_leaks=0"), timeout=300)
    assert "ok" in r.stdout
