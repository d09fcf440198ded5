"""The offline graph builder's attribute-aware pass (input preparation, not
the search path): quantile coordinates, the attribute distance, threshold
candidates against brute force, and the invariants of the assembled rows."""
import numpy as np
import pytest
import torch

from workloads import gen, graph


def test_attribute_quantiles_ties_and_float_columns():
    a = np.array([[5, 0], [1, 0], [5, 0], [9, 0]], dtype=np.int32)
    a[:, 1] = gen.f32_bits([0.5, -2.0, 3.0, -0.0])
    q = graph.attribute_quantiles(a, [gen.ATTR_I32, gen.ATTR_F32])
    # column 0: ranks 2, 1, 2.5 (tie), 4 -> mid-ranks 2.5, 1, 2.5, 4
    np.testing.assert_allclose(q[:, 0], (np.array([2.5, 1.0, 2.5, 4.0]) - 0.5) / 4)
    # float column ranked by value (-2 < -0 < 0.5 < 3), not by bit pattern
    np.testing.assert_allclose(q[:, 1], (np.array([3.0, 1.0, 4.0, 2.0]) - 0.5) / 4)


def _small(n=700, d=8, m=2, seed=3):
    g = np.random.default_rng(seed)
    x = g.normal(size=(n, d)).astype(np.float32)
    a = g.integers(0, 50, size=(n, m)).astype(np.int32)
    return x, a


def test_threshold_candidates_match_brute_force():
    x, a = _small()
    n = x.shape[0]
    X = torch.from_numpy(x).double()
    QA = torch.from_numpy(graph.attribute_quantiles(a, [0, 0]))
    levels = (0.01, 0.1)
    thr = graph._thresholds(QA, levels, seed=1, chunk=128)
    du, cand, du_l, cand_l = graph.candidates(X, 12, QA, thr, 6, chunk=128)
    xd = x.astype(np.float64)
    D = ((xd[:, None, :] - xd[None, :, :]) ** 2).sum(-1)
    np.fill_diagonal(D, np.inf)
    qa = QA.numpy()
    A = np.abs(qa[:, None, :] - qa[None, :, :]).max(-1)
    for i in range(0, n, 37):
        o = np.lexsort((np.arange(n), D[i]))[:12]
        assert cand[i].tolist() == o.tolist()
        for li in range(len(levels)):
            Dm = np.where(A[i] > thr[i, li].item(), np.inf, D[i])
            o = np.lexsort((np.arange(n), Dm))[:6]
            fin = np.isfinite(Dm[o])
            got_d = du_l[li, i].numpy()
            assert np.array_equal(np.isfinite(got_d), fin)
            assert cand_l[li, i][torch.from_numpy(fin)].tolist() == o[fin].tolist()
            # every finite candidate lies within the point's threshold
            assert (A[i][cand_l[li, i][torch.from_numpy(fin)].numpy()] <= thr[i, li].item()).all()


def test_attribute_graph_rows_are_valid_and_reachable():
    x, a = _small(n=1500, d=16)
    R = 16
    adj, entry = graph.build_graph(x, R, "cpu", attrs=a, attr_dtypes=[0, 0])
    n = x.shape[0]
    assert adj.shape == (n, R) and adj.dtype == np.uint32
    for i in range(n):
        row = adj[i][adj[i] != graph.PAD].astype(np.int64)
        assert i not in row
        assert len(set(row.tolist())) == len(row)
        assert (row < n).all()
    assert graph._reachable(n, adj, entry).all()


def test_attribute_edges_raise_valid_neighbour_share():
    # points whose attributes are close should link to each other more often
    # than the vector-only graph links them
    x, a = _small(n=1500, d=16, m=1, seed=5)
    R = 16
    adj_v, _ = graph.build_graph(x, R, "cpu")
    adj_a, _ = graph.build_graph(x, R, "cpu", attrs=a, attr_dtypes=[0])

    def near_share(adj):
        src = np.repeat(np.arange(len(adj)), R)
        dst = adj.reshape(-1)
        ok = dst != graph.PAD
        return float((np.abs(a[src[ok], 0] - a[dst[ok].astype(np.int64), 0]) <= 1).mean())

    assert near_share(adj_a) > near_share(adj_v) + 0.05


def _clustered(n=3000, d=16, k=12, m=2, seed=11):
    g = np.random.default_rng(seed)
    c = g.normal(scale=8.0, size=(k, d))
    x = (c[g.integers(0, k, size=n)] + g.normal(size=(n, d))).astype(np.float32)
    a = g.integers(0, 100, size=(n, m)).astype(np.int32)
    return x, a


def test_ivf_candidates_with_every_list_probed_are_exact():
    x, a = _clustered()
    X = torch.from_numpy(x).double()
    QA = torch.from_numpy(graph.attribute_quantiles(a, [0, 0]))
    thr = graph._thresholds(QA, (0.01, 0.1), seed=1, chunk=512)
    ref = graph.candidates(X, 10, QA, thr, 6, chunk=512)
    got = graph.candidates_ivf(X, 10, QA, thr, 6, lists=12, nprobe=12, batch_elems=1 << 22)
    for r, g_ in zip(ref, got):
        if r.dtype == torch.int64:
            fin = torch.isfinite(ref[0]) if r.dim() == 2 else torch.isfinite(ref[2])
            assert torch.equal(torch.where(fin, r, -1), torch.where(fin, g_, -1))
        else:
            assert torch.equal(torch.isinf(r), torch.isinf(g_))
            fin = torch.isfinite(r)
            assert torch.allclose(r[fin], g_[fin], rtol=1e-12, atol=1e-9)


def test_ivf_candidates_probing_few_lists():
    x, a = _clustered()
    X = torch.from_numpy(x).double()
    QA = torch.from_numpy(graph.attribute_quantiles(a, [0, 0]))
    thr = graph._thresholds(QA, (0.01, 0.1), seed=1, chunk=512)
    du, cand, _, _ = graph.candidates(X, 10, chunk=512)
    dg, cg, dl, cl = graph.candidates_ivf(X, 10, QA, thr, 6, lists=12, nprobe=3, batch_elems=1 << 22)
    # a restricted search: never closer than the exhaustive one, rank by rank
    assert (dg >= du - 1e-9).all()
    # well-separated clusters: nearly all true neighbours are found
    hit = np.mean([len(set(cand[i].tolist()) & set(cg[i].tolist())) / 10 for i in range(len(x))])
    assert hit > 0.95
    # attribute candidates lie within each point's threshold, sorted, no self
    A = (QA[:, None, :] - QA[None, :, :]).abs().max(-1).values
    for li in range(2):
        fin = torch.isfinite(dl[li])
        rows = torch.arange(len(x))[:, None].expand_as(cl[li])
        assert (A[rows[fin], cl[li][fin]] <= thr[rows[fin], li]).all()
        assert (cl[li][fin] != rows[fin]).all()
        assert (dl[li][:, 1:] >= dl[li][:, :-1]).all()


def test_subset_level_candidates_match_brute_force():
    # random-subset levels: each point's nearest members of a seeded subset
    # (itself excluded), after the attribute levels, sorted by (distance, id)
    x, a = _small(n=600, d=8)
    n = x.shape[0]
    X = torch.from_numpy(x).double()
    QA = torch.from_numpy(graph.attribute_quantiles(a, [0, 0]))
    thr = graph._thresholds(QA, (0.1,), seed=1, chunk=128)
    g = np.random.default_rng(9)
    member = torch.from_numpy(g.random((2, n)) < np.array([[0.05], [0.3]]))
    du, cand, du_l, cand_l = graph.candidates(X, 8, QA, thr, 5, chunk=128, member=member)
    assert du_l.shape == (3, n, 5)
    xd = x.astype(np.float64)
    D = ((xd[:, None, :] - xd[None, :, :]) ** 2).sum(-1)
    np.fill_diagonal(D, np.inf)
    for i in range(0, n, 29):
        for s in range(2):
            Dm = np.where(member[s].numpy()[None, :], D[i][None, :], np.inf)[0]
            o = np.lexsort((np.arange(n), Dm))[:5]
            fin = np.isfinite(Dm[o])
            got = cand_l[1 + s, i][torch.from_numpy(fin)].tolist()
            assert got == o[fin].tolist()
            assert np.array_equal(np.isfinite(du_l[1 + s, i].numpy()), fin)
            assert all(member[s, j] and j != i for j in got)


def test_ivf_subset_levels_with_every_list_probed_are_exact():
    x, a = _clustered(n=2000)
    n = x.shape[0]
    X = torch.from_numpy(x).double()
    member = torch.from_numpy(np.random.default_rng(4).random((2, n)) < np.array([[0.02], [0.2]]))
    ref = graph.candidates(X, 10, None, None, 6, chunk=512, member=member)
    got = graph.candidates_ivf(X, 10, None, None, 6, lists=12, nprobe=12, batch_elems=1 << 22, member=member)
    fin = torch.isfinite(ref[2])
    assert torch.equal(fin, torch.isfinite(got[2]))
    assert torch.equal(torch.where(fin, ref[3], -1), torch.where(fin, got[3], -1))
    assert torch.allclose(ref[2][fin], got[2][fin], rtol=1e-12, atol=1e-9)


def test_graph_rows_hold_subset_and_navigation_edges():
    # with subset levels and the default budgets every row stays within R,
    # is duplicate- and self-free, and the graph is reachable from the entry
    x, a = _clustered(n=2500, d=16, k=20)
    R = 32
    adj, entry = graph.build_graph(x, R, "cpu", attrs=a, attr_dtypes=[0, 0], sub_levels=(0.01, 0.1))
    n = x.shape[0]
    assert adj.shape == (n, R)
    for i in range(0, n, 7):
        row = adj[i][adj[i] != graph.PAD].astype(np.int64)
        assert i not in row and len(set(row.tolist())) == len(row) and (row < n).all()
    assert graph._reachable(n, adj, entry).all()
