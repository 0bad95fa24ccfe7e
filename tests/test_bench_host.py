"""Host logic of bench.py that runs without a GPU: the stored HBM-traffic figure
is used only when it was taken on the current kernel sources, and a multi-GPU
request is refused before anything touches a GPU."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_stored_traffic_follows_the_kernel_hash(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.stored_traffic() is None  # no summary at all
    path = tmp_path / bench.TRAFFIC_JSON
    path.write_text(json.dumps({"kernel_hash": bench.kernel_hash(), "traffic_bytes_per_launch": 123}))
    assert bench.stored_traffic() == 123
    path.write_text(json.dumps({"kernel_hash": "0" * 16, "traffic_bytes_per_launch": 123}))
    assert bench.stored_traffic() is None  # taken on other kernel sources
    path.write_text("{not json")
    assert bench.stored_traffic() is None


def test_kernel_hash_covers_the_kernel_sources(tmp_path, monkeypatch):
    h = bench.kernel_hash()
    assert len(h) == 16 and int(h, 16) >= 0
    for f in bench.KERNEL_SOURCES:
        assert os.path.exists(os.path.join(ROOT, f)), f
    # a change in any listed source changes the hash
    src = tmp_path / "src"
    src.mkdir()
    for f in bench.KERNEL_SOURCES:
        dst = src / f
        dst.parent.mkdir(parents=True, exist_ok=True)
        dst.write_bytes(open(os.path.join(ROOT, f), "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(src))
    assert bench.kernel_hash() == h
    last = src / bench.KERNEL_SOURCES[-1]
    last.write_bytes(last.read_bytes() + b"\n")
    assert bench.kernel_hash() != h


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""
