"""Host-side logic of bench.py: the refusal of more than one GPU and the rule that a
counter traffic record is reported only for the kernel sources it was measured on."""
import json
import os
import subprocess
import sys

import bench
from workloads import get

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_traffic_sources_follow_the_gemm_kernel():
    assert bench.traffic_sources(get("qwen3-4b-shape")) == bench.GEMM_SOURCES
    for name in ("qwen3-8b-shape-b8", "qwen3-14b-shape-b16"):
        srcs = bench.traffic_sources(get(name))
        assert srcs == bench.MID_SOURCES and srcs[-1].endswith("gemm_mid.hip")


def _record(tmp_path, name, sha):
    prof = tmp_path / "profiles"
    prof.mkdir(exist_ok=True)
    rec = {"kernel": bench.DOMINANT, "workload": name, "source_sha256": sha, "bytes_per_launch": 12345}
    (prof / f"{bench.DOMINANT}_{name}_traffic.md").write_text("# summary\n\ntraffic-json: " + json.dumps(rec) + "\n")


def test_traffic_record_needs_matching_sources(tmp_path, monkeypatch):
    wl = get("qwen3-14b-shape-b16")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "gemm_source_hash", lambda sources=bench.GEMM_SOURCES: "h-" + sources[-1])
    assert bench.measured_traffic(wl) is None                      # no record
    _record(tmp_path, wl.name, "h-" + bench.GEMM_SOURCES[-1])      # hashed without gemm_mid.hip
    assert bench.measured_traffic(wl) is None
    _record(tmp_path, wl.name, "h-" + bench.MID_SOURCES[-1])
    assert bench.measured_traffic(wl) == 12345


def test_committed_traffic_records_are_well_formed():
    prof = os.path.join(ROOT, "profiles")
    names = [f for f in os.listdir(prof) if f.startswith(bench.DOMINANT) and f.endswith("_traffic.md")]
    assert names
    for f in names:
        recs = [json.loads(line.split(":", 1)[1]) for line in open(os.path.join(prof, f))
                if line.startswith("traffic-json:")]
        assert len(recs) == 1, f
        r = recs[0]
        assert f == f"{bench.DOMINANT}_{r['workload']}_traffic.md"
        assert r["bytes_per_launch"] == r["fetch_bytes_per_launch"] + r["write_bytes_per_launch"]
        # HBM bytes at or above the algorithmic bytes, and no gross re-reads
        assert 1.0 <= r["bytes_per_launch"] / r["algorithmic_bytes_per_launch"] < 1.1, f
