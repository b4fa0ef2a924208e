"""Host-side logic of bench.py (no GPU needed).

bench.py refuses more than one GPU with a message, and reports HBM traffic
only while the kernel and launch sources still hash to the value the
rocprofv3 counters were taken on.
"""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_kernel_hash_ignores_comments_and_whitespace(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("int f() { return 1; }  // one\n/* block */\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", ["k.hip"])
    h = bench.kernel_hash()
    src.write_text("int f()   {\n  return 1;\n}  // another comment\n")
    assert bench.kernel_hash() == h
    src.write_text("int f() { return 2; }\n")
    assert bench.kernel_hash() != h


def test_traffic_only_for_the_profiled_source(tmp_path, monkeypatch):
    f = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    h = bench.kernel_hash()
    f.write_text(json.dumps({"w": {"kernel_hash": h, "traffic_over_alg": 1.001}}))
    assert bench.load_traffic("w", 1000.0) == 1001
    assert bench.load_traffic("other", 1000.0) is None
    f.write_text(json.dumps({"w": {"kernel_hash": "0" * 16, "traffic_over_alg": 1.001}}))
    assert bench.load_traffic("w", 1000.0) is None
    f.write_text("not json")
    assert bench.load_traffic("w", 1000.0) is None


def test_committed_traffic_is_well_formed():
    """Every entry of profiles/traffic.json names its source hash and a
    measured traffic close to the algorithmic bytes."""
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as fh:
        data = json.load(fh)
    assert data
    for e in data.values():
        assert len(e["kernel_hash"]) == 16
        assert 0.999 < e["traffic_over_alg"] < 1.01
        assert e["traffic_bytes_per_launch"] > 0 and e["alg_bytes_per_launch"] > 0


def test_cpu_baseline_runs_on_one_core():
    """The oracle leg pins its thread to one CPU for the timed work and puts
    the affinity back afterwards."""
    from seedgen import workloads as wl
    w = wl.scaled(wl.WORKLOADS[2], [4099])
    before = os.sched_getaffinity(0)
    out = bench.cpu_baseline(w, seconds=0.05)
    assert os.sched_getaffinity(0) == before
    assert out["cores"] == 1 and out["kind"] == "oracle" and out["value"] > 0
    assert "pinned to CPU" in out["sample"]
