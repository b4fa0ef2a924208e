"""The C ABI used from plain C++ (tests/native/cabi_smoke.cpp, built by
__graft_entry__.build()): one scheduled step through librip with HIP's own
runtime and no Python in the loop, checked against exact closed-form values."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "cabi_smoke")


def test_native_cabi_consumer():
    assert os.path.exists(BIN), "tests/native/cabi_smoke is not built; run __graft_entry__.build()"
    print("case native C-ABI smoke", flush=True)
    res = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    print(res.stdout, res.stderr, flush=True)
    assert res.returncode == 0
    assert "cabi smoke ok" in res.stdout


BENCH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                     "paper_1909_08029_amd", "rip_bench_native")


@pytest.mark.parametrize("args", [
    ["--replicas", "8", "--params", "100003", "--group", "4"],
    ["--replicas", "6", "--params", "65537", "--group", "3", "--momentum", "0.9", "--bf16"],
    ["--replicas", "4", "--params", "4099", "--fixed", "0,1,2"],
])
def test_native_throughput_program_runs(args):
    """The C-ABI-only throughput program completes and reports its figures."""
    import json
    assert os.path.exists(BENCH), "rip_bench_native is not built; run __graft_entry__.build()"
    print(f"case native bench {' '.join(args)}", flush=True)
    res = subprocess.run([BENCH, *args, "--steps", "5", "--warmup", "1"], capture_output=True,
                         text=True, timeout=120)
    print(res.stdout, res.stderr, flush=True)
    assert res.returncode == 0
    d = json.loads(res.stdout.strip().splitlines()[-1])
    assert d["steps"] == 5 and d["value_gbps"] > 0 and d["events_gbps"] > 0
    assert d["host_us_per_call"] > 0
