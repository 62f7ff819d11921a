"""The host-side C and C++ code run under the address and
undefined-behaviour sanitizers (CPU only; host compilers, no device code):
the forest builder and predecessor extraction of ScoreBatch and stack
rescoring (paper_1605_04809_amd/csrc/forest_host.cpp) and every entry point
of the fp64 oracle (oracle/oracle.c), each through a driver in
tests/sanitize/ that also checks what its results must satisfy.  Any
out-of-bounds access, use after free, leak or undefined behaviour aborts the
driver."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _build_and_run(tmp_path, compiler, sources, flags, name):
    if shutil.which(compiler) is None:
        pytest.skip(f"{compiler} not available")
    exe = str(tmp_path / name)
    cmd = [compiler, *SAN, *flags, *[os.path.join(ROOT, s) for s in sources], "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, OMP_NUM_THREADS="2", ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr, r.stderr[-6000:]
    return r.stdout


def test_forest_host_code_under_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, "g++", ["paper_1605_04809_amd/csrc/forest_host.cpp",
                                           "tests/sanitize/forest_driver.cpp"], ["-std=c++17"], "forest_driver")
    assert "forest driver ok" in out


def test_oracle_under_sanitizers(tmp_path):
    out = _build_and_run(tmp_path, "gcc", ["oracle/oracle.c", "tests/sanitize/oracle_driver.c"],
                         ["-std=c11", "-fopenmp", "-lm"], "oracle_driver")
    assert "oracle driver ok" in out
