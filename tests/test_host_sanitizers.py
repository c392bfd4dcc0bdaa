"""Host C/C++ under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The library's host fit (csrc/fit.cpp) and the CPU oracle (oracle/oracle.c)
are each compiled with gcc/g++ and -fsanitize=address,undefined into a
driver program of their own (tests/sanitize/), in a temporary directory,
and run: every call must return what it should, and the sanitizers must
report nothing.  The two programs share no code, as the two sides never do.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}"
    return r


@pytest.mark.skipif(shutil.which("g++") is None, reason="no host compiler")
def test_fit_under_sanitizers(tmp_path):
    exe = str(tmp_path / "fit_driver")
    _run(["g++", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "include"),
          os.path.join(ROOT, "tests", "sanitize", "fit_driver.cpp"),
          os.path.join(ROOT, "paper_2202_00441_amd", "csrc", "fit.cpp"), "-o", exe, "-lm"])
    r = _run([exe], env=ENV, timeout=600)
    assert "0 failure(s)" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no host compiler")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-std=c11", *SAN, "-ffp-contract=off",
          os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"),
          os.path.join(ROOT, "oracle", "oracle.c"), "-o", exe, "-lm", "-lpthread"])
    r = _run([exe], env=ENV, timeout=600)
    assert "0 failure(s)" in r.stdout
