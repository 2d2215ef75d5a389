"""Host logic of bench.py (no GPU): the one-GPU rule, the byte model of an
update, and when measured HBM traffic may be reported."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_traffic_needs_the_current_sources_and_options(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path))
    d = {"source_digest": bench.source_digest(), "bench_args": [], "hbm_bytes_per_launch": 123.0}
    (tmp_path / "traffic_k_x_hogwild_netflix.json").write_text(json.dumps(d))
    assert bench.measured_traffic("k_x_hogwild_netflix", []) == 123.0
    assert bench.measured_traffic("k_x_hogwild_netflix", ["--depth", "4"]) is None
    assert bench.measured_traffic("k_y_hogwild_netflix", []) is None
    d["source_digest"] = "0" * 16
    (tmp_path / "traffic_k_x_hogwild_netflix.json").write_text(json.dumps(d))
    assert bench.measured_traffic("k_x_hogwild_netflix", []) is None


def test_source_digest_covers_the_kernel_sources():
    a = bench.source_digest()
    assert a == bench.source_digest() and len(a) == 16
