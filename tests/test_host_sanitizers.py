"""The launch planner (host code, no HIP) compiled with g++ under the
undefined-behaviour and address sanitizers and driven with random and
extreme arguments (tests/plan_fuzz_driver.cpp): any overflow, division by
zero or out-of-bounds access aborts the driver."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2302_07594_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="no host C++ compiler")
def test_planner_under_sanitizers(tmp_path):
    exe = tmp_path / "plan_fuzz"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=undefined,address",
           "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "igemm_plan.cpp"), os.path.join(ROOT, "tests", "plan_fuzz_driver.cpp"),
           "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True)
    env = dict(os.environ, UBSAN_OPTIONS="print_stacktrace=1",
               ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    assert "runtime error" not in r.stderr, r.stderr[-3000:]
    assert r.stdout.startswith("ok ")


def _preload_runtime():
    """The ASan runtime of the host gcc (the sanitized oracle needs it loaded
    first in the Python process that calls it)."""
    r = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no host C compiler")
def test_oracle_pins_under_sanitizers(tmp_path):
    """Every oracle pin set (GEMM, convolution, int16-output update, and the
    planted-mutant checks' unmodified copy) run against the oracle built with
    -fsanitize=address,undefined: an out-of-bounds access, a signed overflow
    or a bad shift in any oracle function aborts the child process."""
    import sys

    from oracle import build as oracle_build
    rt = _preload_runtime()
    if rt is None:
        pytest.skip("gcc's libasan.so not found")
    lib = oracle_build.build_sanitized(str(tmp_path / "liboracle_san.so"))
    env = dict(os.environ, IGEMM_ORACLE_LIB=lib, LD_PRELOAD=rt, OMP_NUM_THREADS="4",
               ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    tests = [os.path.join(ROOT, "tests", t) for t in
             ("test_oracle.py", "test_conv_oracle.py", "test_srs_oracle.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu"] + tests,
                       capture_output=True, text=True, env=env, timeout=900, cwd=ROOT)
    out = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, out
    assert "runtime error" not in r.stderr, out
    assert "AddressSanitizer" not in r.stderr, out
    assert " passed" in r.stdout, out
