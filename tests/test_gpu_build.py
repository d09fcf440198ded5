"""Index construction inside the library (adjacency = NULL, entry = -1).

The library computes the entry point s (the medoid, Alg. 2) and builds the
graph (Sec. II "Graph construction": alpha-pruned exact nearest neighbours,
reverse edges, connectivity repair from s). Checked against what holds
independently of its code:
  - the medoid is the point nearest the float64 centroid (numpy);
  - every row holds valid, distinct ids other than its own;
  - every point is reachable from s;
  - every sampled point's row holds its exact nearest neighbour (float64
    brute force): the nearest candidate is never pruned (nothing is kept
    before it), so a wrong candidate scan shows here;
and the search over the built index (through the C ABI) equals the CPU
oracle searching the same graph, exported with boa_get_graph.
"""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _boa():
    import paper_2609_16175_amd as boa
    return boa


def _nn_rows_ok(x, adj, sample):
    """For each sampled point: its row holds a point at its exact nearest
    distance (float64; near-ties within 1e-5 relative allowed). Returns the
    sampled points whose row does not."""
    dev = torch.device("cuda:0")
    X = torch.from_numpy(x).to(dev).double()
    xn = (X * X).sum(1)
    bad = []
    for s0 in range(0, len(sample), 256):
        ids_np = sample[s0:s0 + 256]
        ids = torch.from_numpy(ids_np).to(dev)
        # candidates by the norm expansion, then exact float64 distances of
        # the 16 nearest by the direct form (the expansion cancels for near points)
        approx = xn[ids][:, None] + xn[None, :] - 2.0 * (X[ids] @ X.T)
        approx[torch.arange(len(ids), device=dev), ids] = float("inf")
        cand = torch.topk(approx, min(16, X.shape[0] - 1), dim=1, largest=False).indices
        exact = ((X[ids][:, None, :] - X[cand]) ** 2).sum(-1)
        best = exact.min(1).values.cpu().numpy()
        for j, u in enumerate(ids_np):
            row = adj[u][adj[u] != 0xFFFFFFFF].astype(np.int64)
            if not len(row):
                bad.append(int(u))
                continue
            dr = ((x[row].astype(np.float64) - x[u].astype(np.float64)) ** 2).sum(1)
            if dr.min() > best[j] * (1 + 1e-5) + 1e-12:
                bad.append(int(u))
    return bad


def _attr_level0_ok(attrs, types, x, adj, sample, q=0.001):
    """The attribute-aware pass of the tightest level (JAG threshold
    pruning): for each sampled point u, the nearest point (float64) among
    those within u's attribute threshold is in u's row. The threshold is
    recomputed here with numpy from its definition: ranks = number of
    strictly smaller values per column (float32 columns as floats), the
    attribute distance = the largest rank gap over the columns, the
    threshold = the ceil(q S)-th smallest distance to the S = min(4096, n)
    points floor(i n / S)."""
    from workloads import gen
    n, m = attrs.shape
    rk = np.empty((n, m), dtype=np.int64)
    for j in range(m):
        col = gen.cells_as_f32(attrs[:, j]) if types[j] == gen.ATTR_F32 else attrs[:, j]
        rk[:, j] = np.searchsorted(np.sort(col), col, side="left")
    S = min(4096, n)
    smp = (np.arange(S, dtype=np.int64) * n) // S
    idx = max(0, int(np.ceil(q * S)) - 1)
    bad = []
    for u in sample:
        t = np.sort(np.abs(rk[smp] - rk[u]).max(1))[idx]
        gap = np.abs(rk - rk[u]).max(1)
        within = np.flatnonzero(gap <= t)
        within = within[within != u]
        if not len(within):
            continue
        dd = ((x[within].astype(np.float64) - x[u].astype(np.float64)) ** 2).sum(1)
        best = dd.min()
        row = adj[u][adj[u] != 0xFFFFFFFF].astype(np.int64)
        rd = ((x[row].astype(np.float64) - x[u].astype(np.float64)) ** 2).sum(1)
        inrow = np.isin(row, within)
        if not inrow.any() or rd[inrow].min() > best * (1 + 1e-5) + 1e-12:
            bad.append(int(u))
    return bad


def _check_graph(x, adj, entry, R):
    from workloads import graph
    n = x.shape[0]
    assert adj.shape == (n, R)
    pad = adj == 0xFFFFFFFF
    safe = np.where(pad, 0, adj).astype(np.int64)
    assert (safe < n).all(), "id out of range"
    assert not ((safe == np.arange(n)[:, None]) & ~pad).any(), "a row holds its own id"
    srt = np.sort(np.where(pad, -1 - np.arange(R)[None, :], safe), axis=1)
    assert not (srt[:, 1:] == srt[:, :-1]).any(), "a row holds an id twice"
    assert (~pad).sum(1).min() >= 1, "a point without out-edges"
    assert graph._reachable(n, adj, entry).all(), "points unreachable from the entry point"
    # the medoid: nearest point to the float64 centroid (independent numpy)
    want = graph.entry_point(x)
    if want != entry:
        c = x.astype(np.float64).mean(0)
        dw = ((x[want].astype(np.float64) - c) ** 2).sum()
        de = ((x[entry].astype(np.float64) - c) ** 2).sum()
        assert abs(de - dw) <= 1e-9 * max(dw, 1e-30), (entry, want)


def _parity(ix_gpu, x, attrs, types, q, r, wl, adj, entry, sample=None, **kw):
    orc = oracle.Index(x, attrs, types, adj, entry)
    sel = np.arange(q.shape[0]) if sample is None else sample
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(orc, q[sel], r[sel], wl.k, sched, threads=8)
    dev = torch.device("cuda:0")
    out = ix_gpu.search(torch.from_numpy(q).to(dev), torch.from_numpy(r).to(dev), k=wl.k, L0=wl.L0, Lmax=wl.Lmax,
                        counters=True, **kw)
    torch.cuda.synchronize()
    got = (out.ids.cpu().numpy().view(np.uint32)[sel], out.dists.cpu().numpy()[sel], out.final_L.cpu().numpy()[sel],
           out.expansions.cpu().numpy()[sel], out.scored.cpu().numpy()[sel])
    for name, a, b in zip(("ids", "dists", "final_L", "expansions", "scored"), got,
                          (ref.ids, ref.dists, ref.final_L, ref.expansions, ref.scored)):
        assert np.array_equal(a, b), f"{name} differ from the oracle on the library-built graph"


def test_tiny_built_in_library():
    from workloads import gen
    wl = gen.TINY
    d = gen.generate(wl)
    types = np.array(wl.attr_dtypes, dtype=np.int32)
    ix = _boa().Index(d.vectors, d.attrs, types, None, -1, R=wl.R)
    adj, entry, repaired = ix.graph()
    _check_graph(d.vectors, adj, entry, wl.R)
    assert repaired >= 0
    assert not _nn_rows_ok(d.vectors, adj, np.arange(wl.n))
    assert not _attr_level0_ok(d.attrs, types, d.vectors, adj, np.arange(0, wl.n, 7))
    for mode in ({}, {"fused": True}, {"split": True}):
        _parity(ix, d.vectors, d.attrs, types, d.queries, d.ranges, wl, adj, entry, **mode)
    ix.close()


@pytest.mark.parametrize("name", ["deep-like-1M-d96", "u8-10M-d128"])
def test_100k_built_in_library(name):
    """100,000 points of the float32 (d = 96, R = 64, a float32 attribute
    column) and uint8 (d = 128, R = 32) recipes."""
    from workloads import gen
    wl = gen.BY_NAME[name].scaled(100_000, nq=2000)
    d = gen.generate(wl)
    types = np.array(wl.attr_dtypes, dtype=np.int32)
    ix = _boa().Index(d.vectors, d.attrs, types, None, -1, R=wl.R)
    adj, entry, repaired = ix.graph()
    _check_graph(d.vectors, adj, entry, wl.R)
    sample = np.sort(np.random.default_rng(3).choice(wl.n, 1000, replace=False))
    bad = _nn_rows_ok(d.vectors, adj, sample)
    assert not bad, f"{len(bad)} sampled rows miss their nearest neighbour (first {bad[:5]})"
    bad = _attr_level0_ok(d.attrs, types, d.vectors, adj, sample[:300])
    assert not bad, f"{len(bad)} sampled rows miss their nearest attribute-close point (first {bad[:5]})"
    qs = np.sort(np.random.default_rng(4).choice(wl.nq, 200, replace=False))
    _parity(ix, d.vectors, d.attrs, types, d.queries, d.ranges, wl, adj, entry, sample=qs, split=True)
    ix.close()


def test_vector_only_build_and_build_params():
    """attr_levels = 0: the graph from vector distances only; alpha = 1
    (the plain relative-neighbourhood rule) keeps fewer edges than 1.2."""
    from workloads import gen
    wl = gen.TINY
    d = gen.generate(wl)
    types = np.array(wl.attr_dtypes, dtype=np.int32)
    boa = _boa()
    edges = {}
    for alpha in (1.0, 1.2):
        ix = boa.Index(d.vectors, d.attrs, types, None, -1, R=wl.R, alpha=alpha, attr_levels=0)
        adj, entry, _ = ix.graph()
        _check_graph(d.vectors, adj, entry, wl.R)
        assert not _nn_rows_ok(d.vectors, adj, np.arange(0, wl.n, 5))
        edges[alpha] = int((adj != 0xFFFFFFFF).sum())
        _parity(ix, d.vectors, d.attrs, types, d.queries, d.ranges, wl, adj, entry, split=True)
        ix.close()
    assert edges[1.0] < edges[1.2]
    with pytest.raises(boa.BoaError):
        boa.Index(d.vectors, d.attrs, types, None, -1, R=wl.R, alpha=0.5)


def test_single_point_and_tiny_n():
    """n = 1 (no edges) and n = 5 (fewer points than 2R candidates)."""
    boa = _boa()
    for n in (1, 5):
        x = np.arange(n * 4, dtype=np.float32).reshape(n, 4)
        a = np.zeros((n, 1), dtype=np.int32)
        ix = boa.Index(x, a, np.zeros(1, np.int32), None, -1, R=8)
        adj, entry, _ = ix.graph()
        assert entry == (n - 1) // 2 if n > 1 else entry == 0
        if n > 1:
            from workloads import graph
            assert graph._reachable(n, adj, entry).all()
        q = torch.from_numpy(x[:1].copy()).to("cuda:0")
        r = torch.from_numpy(np.array([[[0, 0]]], dtype=np.int32)).to("cuda:0")
        out = ix.search(q, r, k=1, fixed_L=8)   # wider than n: exhaustive
        torch.cuda.synchronize()
        assert out.ids.cpu().numpy()[0, 0] == 0
        ix.close()
