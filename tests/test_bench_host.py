"""Host-side contract of bench.py that needs no GPU: the one-GPU refusal, and
when the recorded HBM traffic of the attention kernel is reported (only for
the kernel sources and workload the counters were taken with)."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_source_hash_ignores_comments_and_blank_lines(tmp_path, monkeypatch):
    a, b, c = tmp_path / "a.hip", tmp_path / "b.hip", tmp_path / "c.hip"
    a.write_text("int f() {\n  return 1;  // one\n}\n")
    b.write_text("// header\n\nint f() {\n  return 1;\n}\n\n")
    c.write_text("int f() {\n  return 2;\n}\n")
    monkeypatch.setattr(bench, "ATTN_SOURCES", [str(a)])
    ha = bench.attn_source_hash()
    monkeypatch.setattr(bench, "ATTN_SOURCES", [str(b)])
    assert bench.attn_source_hash() == ha
    monkeypatch.setattr(bench, "ATTN_SOURCES", [str(c)])
    assert bench.attn_source_hash() != ha


def test_recorded_traffic_only_for_matching_sources_and_workload(tmp_path, monkeypatch):
    rec = {"workload": "w1", "source_sha256": bench.attn_source_hash(), "read_bytes": 1000, "write_bytes": 24}
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC", str(f))
    assert bench.recorded_traffic("w1") == 1024
    assert bench.recorded_traffic("w2") is None
    f.write_text(json.dumps({**rec, "source_sha256": "0" * 64}))
    assert bench.recorded_traffic("w1") is None
    monkeypatch.setattr(bench, "TRAFFIC", str(tmp_path / "missing.json"))
    assert bench.recorded_traffic("w1") is None
