"""Host-side pieces of bench.py that need no GPU."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]


def test_doubling_widths():
    assert bench.doubling_widths(16, 512) == [16, 32, 64, 128, 256, 512]
    assert bench.doubling_widths(16, 1024)[-1] == 1024
    assert bench.doubling_widths(10, 100) == [10, 20, 40, 80, 100]
    assert bench.doubling_widths(16, 16) == [16]


def test_recorded_traffic_follows_the_source_digest(tmp_path, monkeypatch):
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    key = next(iter(rec))
    entry = rec[key]
    # the committed record is used only while its digest matches the sources
    want = float(entry["traffic_bytes_per_launch"]) if entry["source_sha256"] == bench.source_digest() else None
    assert bench.recorded_traffic(key) == want
    assert bench.recorded_traffic("no-such-workload/split/1..1") is None
    # a stale digest disables the figure
    (tmp_path / "profiles").mkdir()
    stale = {key: dict(entry, source_sha256="0" * 64)}
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps(stale))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_digest", lambda: "f" * 64)
    assert bench.recorded_traffic(key) is None


def test_selectivity_summary():
    import numpy as np
    n, k = 1000, 10
    n_valid = np.array([0, 5, 10, 50, 500, 1000], dtype=np.int64)
    rq = np.array([1.0, 0.5, 1.0, 0.8, 0.9, 1.0])
    s = bench.selectivity_summary(n_valid, n, k, rq)
    assert s["min_valid_points"] == 0 and s["queries_with_fewer_than_k"] == 2
    assert sum(s["histogram"].values()) == len(n_valid)
    # 0 -> first bin; 0.005 and 0.01 -> [1e-3, 1e-2) and [1e-2, 0.03); 1.0 -> last bin
    assert s["histogram"]["0-0.0001"] == 1
    assert s["histogram"]["0.001-0.01"] == 1
    assert s["histogram"]["0.01-0.03"] == 1
    assert s["histogram"]["0.3-1"] == 2
    assert s["recall_by_bin"]["0.3-1"] == 0.95
    assert abs(s["median"] - 0.03) < 1e-12
