"""The host-side code of libt2vattn (tile scheduler, makespan model, argument validation,
cascade planner) under AddressSanitizer, UndefinedBehaviorSanitizer and leak detection:
tests/host_sanitizer_driver.cpp is built with g++ (host code only, no device code) and run;
a canary first shows that the sanitizer reports an out-of-bounds write here."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_01701_amd", "csrc")
FLAGS = ["-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")


def build(sources, out):
    r = subprocess.run(["g++", *FLAGS, "-I", os.path.join(ROOT, "include"), *sources, "-o", out],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]


def test_sanitizer_canary(tmp_path):
    src = tmp_path / "canary.cpp"
    src.write_text("#include <vector>\nint main(int c, char**) { std::vector<int> v(4); v.data()[4 + c] = 1; "
                   "return v[0]; }\n")
    exe = str(tmp_path / "canary")
    build([str(src)], exe)
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=60)
    assert r.returncode != 0 and "AddressSanitizer" in r.stderr


def test_host_code_is_clean_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_sanitizer_driver")
    build([os.path.join(ROOT, "tests", "host_sanitizer_driver.cpp"), os.path.join(CSRC, "t2v_host.cpp"),
           os.path.join(CSRC, "t2v_plan.cpp")], exe)
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=300)
    report = r.stdout[-3000:] + r.stderr[-3000:]
    assert "Sanitizer" not in r.stderr and "runtime error" not in r.stderr, report
    assert r.returncode == 0 and "0 failed checks" in r.stdout, report
