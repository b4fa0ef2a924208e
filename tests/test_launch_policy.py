"""The launch residency policy (paper_1909_08029_amd/csrc/rip_launch_policy.h)
on the CPU: single-shape launches take their table entry, groups above the
specialized sizes use the chunked-path entry, mixed launches take the
byte-weighted mean rounded up to an even cap (tests/native/launch_policy_test.cpp)."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_launch_policy():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "launch_policy_test")
        cmd = ["g++", "-std=c++17", "-O1", "-Wall", "-Werror",
               "-I", os.path.join(ROOT, "paper_1909_08029_amd", "csrc"),
               os.path.join(ROOT, "tests", "native", "launch_policy_test.cpp"), "-o", exe]
        build = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
        assert build.returncode == 0, build.stderr[-3000:]
        res = subprocess.run([exe], capture_output=True, text=True, timeout=60)
        assert res.returncode == 0, (res.stdout, res.stderr[-3000:])
        assert "launch policy ok" in res.stdout
