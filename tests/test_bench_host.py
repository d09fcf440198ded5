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


def test_recall_strict_and_tie_tolerant():
    """Recall verifies every returned id on its own: its predicates, its
    distance recomputed from the vectors, and repeats."""
    import numpy as np
    PAD = 0xFFFFFFFF
    k = 3
    # points on one axis, queries at the origin: squared distance = x^2
    x = np.array([7, 1, 2, 3, 8, 1, 2, 10, 11, 3, 3, 12], dtype=np.float32)
    X = np.zeros((12, 4), dtype=np.float32)
    X[:, 0] = x
    a = np.zeros((12, 1), dtype=np.int32)
    a[[5, 6], 0] = 1
    a[10, 0] = 5
    Q = np.zeros((3, 4), dtype=np.float32)
    ranges = np.array([[[0, 0]], [[1, 1]], [[100, 200]]], dtype=np.int32)
    gt_ids = np.array([[1, 2, 3], [5, 6, -1], [0, 0, 0]], dtype=np.int64)
    gt_d = np.array([[1.0, 4.0, 9.0], [1.0, 4.0, np.inf], [np.inf, np.inf, np.inf]])
    n_valid = np.array([9, 2, 0])

    def rec(ids, per_query=False):
        ver = bench.verified_rows(ids, X, Q, a, ranges, (0,))
        return bench.recall(ids, gt_ids, gt_d, n_valid, k, ver, per_query=per_query)

    # query 0: ids 1, 2 right, 9 wrong but tied with the 3rd exact distance
    # query 1: both valid points found, then padding
    # query 2: no valid point, nothing returned
    ids = np.array([[1, 2, 9], [6, 5, PAD], [PAD, PAD, PAD]], dtype=np.uint32)
    strict, tie = rec(ids)
    assert abs(strict - (2 / 3 + 1 + 1) / 3) < 1e-12
    np.testing.assert_allclose(rec(ids, True), [1.0, 1.0, 1.0])
    assert abs(tie - 1.0) < 1e-12
    # a farther wrong id is not forgiven
    ids2 = ids.copy()
    ids2[0, 2] = 4
    assert abs(rec(ids2, True)[0] - 2 / 3) < 1e-12
    # an id that violates its query's predicate counts for nothing, even at
    # the tied distance
    ids3 = ids.copy()
    ids3[0, 2] = 10
    assert abs(rec(ids3, True)[0] - 2 / 3) < 1e-12
    # a repeated id counts once
    ids4 = ids.copy()
    ids4[0] = [1, 1, 2]
    assert abs(rec(ids4, True)[0] - 2 / 3) < 1e-12
    s4, _ = rec(ids4)
    assert abs(s4 - (2 / 3 + 1 + 1) / 3) < 1e-12
    # returning an id where no point is valid scores 0
    ids5 = ids.copy()
    ids5[2, 0] = 3
    assert rec(ids5, True)[2] == 0.0


def test_exact_filtered_topk_matches_brute_force():
    import numpy as np
    import torch
    from workloads import gen
    g = np.random.default_rng(7)
    n, d, nq, k = 400, 12, 20, 5
    X = g.normal(size=(n, d)).astype(np.float32)
    Q = g.normal(size=(nq, d)).astype(np.float32)
    A = np.empty((n, 2), dtype=np.int32)
    A[:, 0] = g.integers(0, 100, size=n)
    A[:, 1] = gen.f32_bits(g.normal(size=n).astype(np.float32))
    R = np.empty((nq, 2, 2), dtype=np.int32)
    lo = g.integers(0, 60, size=nq)
    R[:, 0, 0], R[:, 0, 1] = lo, lo + g.integers(0, 40, size=nq)
    fl = np.sort(g.normal(size=(nq, 2)).astype(np.float32), axis=1)
    R[:, 1, 0], R[:, 1, 1] = gen.f32_bits(fl[:, 0]), gen.f32_bits(fl[:, 1])
    R[0, 0] = [1000, 2000]   # no valid point
    ids, dd, nv = bench.exact_filtered_topk(torch, torch.from_numpy(X), torch.from_numpy(A), {1},
                                            torch.from_numpy(Q), torch.from_numpy(R), k, chunk=7)
    a1 = gen.cells_as_f32(A[:, 1])
    for i in range(nq):
        lo1, hi1 = gen.cells_as_f32(R[i, 1])
        ok = (A[:, 0] >= R[i, 0, 0]) & (A[:, 0] <= R[i, 0, 1]) & (a1 >= lo1) & (a1 <= hi1)
        assert nv[i] == ok.sum()
        dist = ((X.astype(np.float64) - Q[i].astype(np.float64)) ** 2).sum(1)
        dist[~ok] = np.inf
        o = np.lexsort((np.arange(n), dist))[:k]
        fin = np.isfinite(dist[o])
        assert ids[i][fin].tolist() == o[fin].tolist()
        np.testing.assert_allclose(dd[i][fin], dist[o][fin], rtol=1e-12)
        assert np.isinf(dd[i][~fin]).all()
