"""Sanitizer builds of the host code (CPU only): the oracle's C under
AddressSanitizer + UndefinedBehaviorSanitizer, and the request batcher
(csrc/batcher.cpp, with the ensemble entry points it calls replaced by a
stub) under ASan + UBSan and under ThreadSanitizer.  Each driver exercises
its code on small ragged inputs and concurrent callers; any report fails the
test.  Nothing here touches a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", TSAN_OPTIONS="halt_on_error=1",
           OMP_NUM_THREADS="2")


def _build_and_run(tmp_path, compiler, srcs, flags, name):
    exe = str(tmp_path / name)
    cmd = [compiler, *flags, "-g", "-O1", "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"),
           *srcs, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "sanitizer" in (r.stderr or "").lower() and "not found" in r.stderr.lower():
        pytest.skip(f"{name}: this toolchain has no such sanitizer runtime")
    assert r.returncode == 0, r.stderr[-3000:]
    run = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=240)
    out = run.stdout + run.stderr
    assert run.returncode == 0 and "ERROR" not in out and "runtime error" not in out, out[-4000:]
    return out


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_asan_ubsan(tmp_path):
    out = _build_and_run(tmp_path, "gcc", [os.path.join(HERE, "oracle_driver.c"), os.path.join(ROOT, "oracle", "fso.c")],
                         ["-std=c11", "-fopenmp", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                          "-ffp-contract=off", "-lm"], "oracle_asan")
    assert "oracle driver ok" in out


# ThreadSanitizer from the ROCm LLVM toolchain: gcc 11's does not intercept
# pthread_cond_clockwait (which libstdc++ uses for condition_variable::
# wait_until) and then reports every timed wait as a double lock.
CLANGXX = "/opt/rocm/llvm/bin/clang++"


@pytest.mark.parametrize("san", ["address,undefined", "thread"])
def test_batcher_under_sanitizers(tmp_path, san):
    cxx = "g++" if san != "thread" else CLANGXX
    if shutil.which(cxx) is None:
        pytest.skip(f"{cxx} not found")
    src = [os.path.join(HERE, "batcher_driver.cpp"), os.path.join(ROOT, "paper_2003_01538_amd", "csrc", "batcher.cpp")]
    flags = ["-std=c++17", "-pthread", f"-fsanitize={san}", "-fno-sanitize-recover=all"]
    out = _build_and_run(tmp_path, cxx, src, flags, "batcher_" + san.split(",")[0])
    assert "batcher driver ok" in out
