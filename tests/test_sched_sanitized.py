"""The group scheduler under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): tests/native/sched_fuzz.cpp links rip_sched.cpp alone, runs
thousands of random configurations of every mode through the C ABI and
checks the schedules' invariants; any memory error or undefined behaviour
aborts the run."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_scheduler_fuzz_under_sanitizers():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "sched_fuzz")
        cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
               "-I", os.path.join(ROOT, "include"),
               "-I", os.path.join(ROOT, "paper_1909_08029_amd", "csrc"),
               os.path.join(ROOT, "tests", "native", "sched_fuzz.cpp"),
               "-x", "c++", os.path.join(ROOT, "paper_1909_08029_amd", "csrc", "rip_sched.cpp"),
               "-o", exe]
        build = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
        assert build.returncode == 0, build.stderr[-3000:]
        # The process environment is passed on unchanged; ASan is told not to
        # insist on being the first library loaded.
        env = dict(os.environ,
                   ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
                   UBSAN_OPTIONS="print_stacktrace=1")
        res = subprocess.run([exe, "3000"], capture_output=True, text=True, timeout=600, env=env)
        assert res.returncode == 0, (res.stdout[-2000:], res.stderr[-4000:])
        assert "sched fuzz ok" in res.stdout
