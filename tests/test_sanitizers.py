"""The CPU code under AddressSanitizer and UndefinedBehaviorSanitizer: the
oracle (oracle/lda_oracle.c) and the host layout planner
(paper_2007_08725_amd/csrc/layout.cpp) are built with -fsanitize=address,undefined
(host compilers only; no device code is involved) and driven over seeded
small corpora by tests/sanitize/*.  Any sanitizer report fails the run."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600, **kw)
    assert r.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), r.stdout[-3000:], r.stderr[-3000:])
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_checks")
    _run(["gcc", "-std=c11", "-ffp-contract=off", *SAN, "-I", os.path.join(ROOT, "oracle"),
          os.path.join(HERE, "sanitize", "oracle_checks.c"), os.path.join(ROOT, "oracle", "lda_oracle.c"),
          "-lm", "-o", exe])
    r = _run([exe], env=ENV)
    assert "oracle checks passed" in r.stdout


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="g++ or the HIP headers are not installed")
def test_layout_planner_under_sanitizers(tmp_path):
    exe = str(tmp_path / "layout_checks")
    csrc = os.path.join(ROOT, "paper_2007_08725_amd", "csrc")
    _run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", csrc,
          os.path.join(HERE, "sanitize", "layout_checks.cpp"), os.path.join(csrc, "layout.cpp"), "-o", exe])
    r = _run([exe], env=ENV)
    assert "layout checks passed" in r.stdout
