"""The host-only C++ (planner, owner map, schedule algebra) and the CPU oracle, built
with g++ under AddressSanitizer and UndefinedBehaviorSanitizer and driven on valid and
invalid inputs (tests/sanitize/*.cpp).  A sanitizer report fails the run.  CPU only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
CSRC = os.path.join(ROOT, "paper_2607_03229_amd", "csrc")

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")


def _build_and_run(tmp_path, name, sources, extra=()):
    exe = str(tmp_path / name)
    cmd = (["g++", "-std=c++17", "-O1", "-g"] + SAN + list(extra) + ["-o", exe] + sources)
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="4")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report[-4000:]
    assert "AddressSanitizer" not in report and "runtime error" not in report, report[-4000:]
    return report


def test_host_code_under_sanitizers(tmp_path):
    src = [os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp")] + \
          [os.path.join(CSRC, f) for f in ("plan.cpp", "owner.cpp", "derive.cpp")]
    out = _build_and_run(tmp_path, "host_checks", src)
    assert "host checks passed" in out


def test_oracle_under_sanitizers(tmp_path):
    src = [os.path.join(ROOT, "tests", "sanitize", "oracle_driver.cpp"),
           os.path.join(ROOT, "oracle", "mpipe_ref.cpp")]
    out = _build_and_run(tmp_path, "oracle_checks", src, extra=["-fopenmp"])
    assert "oracle checks passed" in out
