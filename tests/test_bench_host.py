"""Host-side contract of bench.py (no GPU): the one-GPU guard and the
traffic record lookup that feeds `roofline.traffic`."""
import hashlib
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.fixture()
def fake_root(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    (tmp_path / "k.hip").write_text("kernel source v1\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return tmp_path


def _record(root, sha):
    rec = {"kernel": "k", "entry": "attn_bwd_dkdv", "workload": "llama8b", "sources": ["k.hip"],
           "sources_sha256": sha, "fetch_bytes_per_launch": 1000, "write_bytes_per_launch": 24}
    (root / "profiles" / "traffic_k.md").write_text("# summary\n\ntraffic-record: " + json.dumps(rec) + "\n")


def test_traffic_record_matches_current_sources(fake_root):
    _record(fake_root, hashlib.sha256(b"kernel source v1\n").hexdigest())
    assert bench.measured_traffic("attn_bwd_dkdv", "llama8b") == 1024
    assert bench.measured_traffic("attn_bwd_dkdv", "wholedoc") is None
    assert bench.measured_traffic("attn_bwd_dq", "llama8b") is None


def test_traffic_record_is_dropped_when_the_kernel_changed(fake_root):
    _record(fake_root, hashlib.sha256(b"kernel source v1\n").hexdigest())
    (fake_root / "k.hip").write_text("kernel source v2\n")
    assert bench.measured_traffic("attn_bwd_dkdv", "llama8b") is None


def test_committed_records_parse():
    """Every committed record names existing sources; its value is either the
    recorded bytes (sources unchanged) or None (changed since)."""
    import glob
    for path in glob.glob(os.path.join(ROOT, "profiles", "traffic_*.md")):
        lines = [l for l in open(path) if l.startswith("traffic-record:")]
        assert len(lines) == 1, path
        rec = json.loads(lines[0].split(":", 1)[1])
        for src in rec["sources"]:
            assert os.path.exists(os.path.join(ROOT, src)), src
        v = bench.measured_traffic(rec["entry"], rec["workload"])
        assert v is None or v == rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]


def test_planner_study_runs_on_the_host():
    """`bench.py --study planner` needs no GPU: one JSON line per (lengths,
    N, planner), the Llama3 per-sequence plan is the most imbalanced on the
    log-normal lengths and the hybrid meets its target ratio."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--study", "planner",
                        "--seeds", "1"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    rows = [json.loads(x) for x in r.stdout.splitlines() if x.startswith("{")]
    plan_rows = [x for x in rows if x["study"] == "planner"]
    assert len(plan_rows) == 8 * len(bench.PLANNERS)
    for cp in (2, 4, 8, 16, 32):
        by = {x["planner"]: x for x in plan_rows if x["workload"] == "llama8b" and x["cp"] == cp}
        assert by["per_seq"]["imbalance_max"] > by["per_doc"]["imbalance_max"]
        assert by["hybrid"]["imbalance_max"] <= 1.05 + 1e-12
        assert by["whole_lpt"]["recv_tokens_max"] == 0
