"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* csrc/validate.cpp, the library's host-side argument checks, driven by a fuzz harness
  (tests/host/validate_fuzz.cpp) through hostile sizes, pitches, counts, enum values and
  pointers, honouring each check's documented preconditions;
* oracle/cpu_oracle.c, the C oracle, on random BSR matrices with every array allocated to its
  exact size (tests/host/oracle_fuzz.c), checked against a plain loop.

Both are built with g++/gcc (host code only, no GPU code) and must run clean: any sanitizer
report aborts the program with a non-zero status.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
ENV = dict(os.environ, ASAN_OPTIONS="verify_asan_link_order=0:detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _build_and_run(cmd, exe):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=600)
    assert r.returncode == 0 and r.stdout.startswith("ok"), (r.stdout[-2000:] + r.stderr[-4000:])
    return r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_validation_under_sanitizers(tmp_path):
    exe = str(tmp_path / "validate_fuzz")
    out = _build_and_run(["g++", "-std=c++17", *SAN,
                          "-I", os.path.join(ROOT, "paper_2106_08846_amd", "csrc"),
                          os.path.join(ROOT, "tests", "host", "validate_fuzz.cpp"),
                          os.path.join(ROOT, "paper_2106_08846_amd", "csrc", "validate.cpp"),
                          "-o", exe], exe)
    batches = int(out.split()[3])
    assert batches > 100, "the fuzz must reach the cross-product checks"


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_c_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_fuzz")
    _build_and_run(["gcc", "-std=c11", *SAN,
                    os.path.join(ROOT, "tests", "host", "oracle_fuzz.c"),
                    os.path.join(ROOT, "oracle", "cpu_oracle.c"), "-o", exe, "-lm"], exe)
