"""bench.py's command-line contract that does not need a GPU."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_is_null_when_the_copy_source_changed(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    p = tmp_path / "traffic_kv_copy_store_w.txt"
    p.write_text(f"source_digest={bench._src_digest()}\ntraffic_bytes_per_launch=123\n")
    assert bench._load_traffic("kv_copy_store", "w") == 123.0
    p.write_text("source_digest=0000\ntraffic_bytes_per_launch=123\n")
    assert bench._load_traffic("kv_copy_store", "w") is None
    assert bench._load_traffic("kv_copy_store", "absent") is None
