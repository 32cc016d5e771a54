"""bench.py's host-side contract (no GPU): more than one GPU is refused with a
message, and the committed window-pass traffic summary is read only while
the kernel sources match the profiled ones."""
import os
import subprocess
import sys

from conftest import ROOT


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_summary_follows_the_sources(monkeypatch, tmp_path):
    sys.path.insert(0, ROOT)
    import bench
    h = bench.window_source_hash()
    assert len(h) == 16
    f = tmp_path / "traffic.md"
    f.write_text(f"traffic_bytes_per_launch: 123456\nsource_hash: {h}\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.committed_traffic() == 123456.0
    f.write_text("traffic_bytes_per_launch: 123456\nsource_hash: 0000000000000000\n")
    assert bench.committed_traffic() is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.md"))
    assert bench.committed_traffic() is None
