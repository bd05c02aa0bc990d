"""CPU checks of bench.py's contract pieces that need no GPU: the one-GPU guard and the
traffic record (valid only for the kernel sources it was taken on)."""
import json
import os
import subprocess
import sys

import bench
from paper_2609_36301_amd.inputs import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_committed_traffic_records_parse():
    # each committed record is well formed; bench.py uses it only while the sources match
    for name in ("teaser_prefill", "mid"):
        path = os.path.join(ROOT, "profiles", "route_%s_traffic.md" % name)
        lines = [l for l in open(path) if l.startswith("traffic-record:")]
        assert len(lines) == 1
        rec = json.loads(lines[0].split(":", 1)[1])
        assert rec["workload"] == name and len(rec["source_sha256"]) == 64
        assert rec["fetch_kib_per_call"] > 0 and rec["fetch_scale"] > 0
        t = bench.measured_traffic(WORKLOADS[name])
        assert t is None or t > 0
    assert bench.measured_traffic(WORKLOADS["tiny"]) is None  # no record for this workload


def test_traffic_record_is_dropped_when_sources_change(tmp_path, monkeypatch):
    w = WORKLOADS["teaser_prefill"]
    prof = tmp_path / "profiles"
    prof.mkdir()
    rec = {"workload": w.name, "source_sha256": "0" * 64, "fetch_kib_per_call": 100.0,
           "write_kib_per_call": 10.0, "fetch_scale": 2.0, "write_scale": 1.0}
    (prof / ("route_%s_traffic.md" % w.name)).write_text("x\ntraffic-record: %s\n" % json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 64)
    assert bench.measured_traffic(w) == 1024 * (100 * 2 + 10)
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "1" * 64)
    assert bench.measured_traffic(w) is None


def test_replay_split_times_exactly_the_requested_steps():
    for steps in (1, 2, 5, 7, 20, 200, 97):
        reps, per = bench.replay_split(steps)
        assert reps * per == steps and 1 <= reps <= 10
    assert bench.replay_split(20) == (10, 2)
