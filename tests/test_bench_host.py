"""Host-side helpers of bench.py (no GPU): the comment-insensitive source
digest that keys the committed HBM counter summaries, the copy-calibrated
traffic read from them, and the one-GPU guard."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_code_text_ignores_comments_and_whitespace():
    a = "int f(int x) {  // doubles\n  return 2 * x; /* the\n multi-line */ }\n"
    b = "int f(int x) { return 2 * x; }"
    assert bench.code_text(a) == bench.code_text(b)
    assert bench.code_text(a) != bench.code_text(b.replace("2 * x", "3 * x"))


def test_source_digest_keeps_comment_edits_and_sees_code_edits(tmp_path):
    (tmp_path / "k.hip").write_text("__global__ void k(float* p) { p[0] = 1.f; }\n")
    (tmp_path / "h.h").write_text("// header\nconstexpr int kN = 4;\n")
    (tmp_path / "notes.txt").write_text("not a source")
    d0 = bench.source_digest(str(tmp_path))
    (tmp_path / "h.h").write_text("// a longer comment\n\nconstexpr int kN = 4;  // four\n")
    (tmp_path / "notes.txt").write_text("changed")
    assert bench.source_digest(str(tmp_path)) == d0
    (tmp_path / "h.h").write_text("constexpr int kN = 5;\n")
    assert bench.source_digest(str(tmp_path)) != d0


def test_counter_traffic_calibrates_and_rejects_stale_summaries(tmp_path, monkeypatch):
    data = {"source_sha256": bench.source_digest(), "unit": "launch",
            "copy": {"bytes_read": 1 << 20, "bytes_written": 1 << 20,
                     "fetch_kib": 512.0, "write_kib": 1024.0},
            "kernels": {"fwdbwd": {"fetch_kib": 100.0, "write_kib": 50.0, "calls": 3}}}
    path = tmp_path / "hbm_counters_{}.md"
    (tmp_path / "hbm_counters_x.md").write_text("# t\n\n```json\n" + json.dumps(data) + "\n```\n")
    monkeypatch.setattr(bench, "COUNTERS", str(path))
    # FETCH_SIZE counts half the copy's bytes (factor 2), WRITE_SIZE all (factor 1)
    assert bench.counter_traffic("x", "fwdbwd") == 100 * 1024 * 2 + 50 * 1024
    assert bench.counter_traffic("x", "update") is None
    assert bench.counter_traffic("missing", "fwdbwd") is None
    data["source_sha256"] = "0" * 64
    (tmp_path / "hbm_counters_x.md").write_text("```json\n" + json.dumps(data) + "\n```\n")
    assert bench.counter_traffic("x", "fwdbwd") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
