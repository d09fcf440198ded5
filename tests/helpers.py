"""Shared test helpers: small random indexes and independent numpy checks."""
import numpy as np

import oracle
from workloads import gen

PAD = 0xFFFFFFFF
I32_MIN, I32_MAX = -2**31, 2**31 - 1


def ring_knn_graph(x: np.ndarray, R: int, seed: int) -> np.ndarray:
    """kNN rows (float64) with the last slot pointing to i+1: strongly connected."""
    n = x.shape[0]
    xf = x.astype(np.float64)
    sq = (xf * xf).sum(1)
    d = sq[:, None] + sq[None, :] - 2.0 * (xf @ xf.T)
    np.fill_diagonal(d, np.inf)
    order = np.argsort(d, axis=1, kind="stable")[:, :R - 1]
    adj = np.full((n, R), PAD, dtype=np.uint32)
    adj[:, :R - 1] = order
    rng = np.random.default_rng(seed)
    # knock out a few slots to exercise padding in the middle of rows
    holes = rng.random((n, R - 1)) < 0.1
    adj[:, :R - 1][holes] = PAD
    nxt = (np.arange(n) + 1) % n
    for i in range(n):
        if nxt[i] not in adj[i, :R - 1]:
            adj[i, R - 1] = nxt[i]
    return adj


def random_arrays(n=400, d=16, m=2, R=12, dtype="f32", seed=0, f32_col=False):
    """(vectors, attrs, attr_dtypes, adjacency, entry) of a small random index."""
    rng = np.random.default_rng(seed)
    if dtype == "u8":
        x = rng.integers(0, 256, size=(n, d)).astype(np.uint8)
    else:
        c = rng.normal(size=(4, d))
        x = (c[rng.integers(0, 4, n)] + 0.5 * rng.normal(size=(n, d))).astype(np.float32)
    attrs = rng.integers(0, 100, size=(n, m)).astype(np.int32)
    types = np.zeros(m, dtype=np.int32)
    if f32_col:
        types[-1] = gen.ATTR_F32
        attrs[:, -1] = gen.f32_bits(rng.normal(size=n).astype(np.float32))
    adj = ring_knn_graph(x, R, seed)
    return x, attrs, types, adj, int(rng.integers(0, n))


def random_index(**kw):
    return oracle.Index(*random_arrays(**kw))


def random_queries(ix, nq, sel_width, seed, f32_col=False):
    rng = np.random.default_rng(seed + 1)
    n, d = ix.vectors.shape
    if ix.vectors.dtype == np.uint8:
        q = rng.integers(0, 256, size=(nq, d)).astype(np.uint8)
    else:
        q = ix.vectors[rng.integers(0, n, nq)] + 0.3 * rng.normal(size=(nq, d)).astype(np.float32)
        q = q.astype(np.float32)
    r = np.zeros((nq, ix.m, 2), dtype=np.int32)
    lo = rng.integers(0, 100 - sel_width + 1, size=(nq, ix.m))
    r[:, :, 0] = lo
    r[:, :, 1] = lo + sel_width - 1
    if f32_col:
        a = rng.normal(size=(nq, 2)).astype(np.float32)
        r[:, -1, 0] = gen.f32_bits(np.minimum(a[:, 0], a[:, 1]))
        r[:, -1, 1] = gen.f32_bits(np.maximum(a[:, 0], a[:, 1]) + 0.5)
    return q, r


def numpy_valid(ix, r):
    """Eq. 2 evaluated with numpy, column by column in its own type."""
    ok = np.ones(ix.n, dtype=bool)
    for j in range(ix.m):
        if ix.attr_dtypes[j] == gen.ATTR_F32:
            a = gen.cells_as_f32(ix.attrs[:, j])
            lo, hi = gen.cells_as_f32(r[j:j + 1, 0])[0], gen.cells_as_f32(r[j:j + 1, 1])[0]
        else:
            a, lo, hi = ix.attrs[:, j], r[j, 0], r[j, 1]
        ok &= (lo <= a) & (a <= hi)
    return ok


def numpy_filtered_topk(ix, q, r, k):
    """Def. 1 with float64 distances: (ids, d64) of the k nearest valid points."""
    ok = np.flatnonzero(numpy_valid(ix, r))
    d = ((ix.vectors[ok].astype(np.float64) - q.astype(np.float64)) ** 2).sum(1)
    o = np.lexsort((ok, d))[:k]
    return ok[o], d[o]


def assert_same_up_to_near_ties(ids, dists, ref_ids, ref_d64, rel=1e-5):
    """ids equal except where float rounding can swap near-tied neighbours."""
    valid = ids != PAD
    assert valid.sum() == len(ref_ids)
    np.testing.assert_allclose(dists[valid], ref_d64, rtol=1e-5, atol=1e-6)
    for j, (a, b) in enumerate(zip(ids[valid], ref_ids)):
        if a != b:
            # allowed only if a tie partner sits within rel of position j
            near = np.abs(ref_d64 - ref_d64[j]) <= rel * max(ref_d64[j], 1e-30)
            assert a in set(ref_ids[near]) or near.sum() > 1, (j, a, b)




def load_beam_trace(path):
    """The hand-traced golden graph of tests/golden/beam_trace.txt:
    (vectors n x 4 float32, attrs n x 1, adjacency n x 3, entry, queries
    {name: (q, ranges)}, SEARCH cases, BOA cases, WARM cases)."""
    pts, adj, queries, searches, boas, entry = {}, {}, {}, [], [], None
    warms = []
    with open(path) as f:
        for line in f:
            p = line.split()
            if not p or p[0].startswith("#"):
                continue
            if p[0] == "POINT":
                pts[int(p[1])] = (float(p[2]), float(p[3]), int(p[4]))
            elif p[0] == "ADJ":
                adj[int(p[1])] = [PAD if v == "-" else int(v) for v in p[2:]]
            elif p[0] == "ENTRY":
                entry = int(p[1])
            elif p[0] == "QUERY":
                queries[p[1]] = (np.array([[float(p[2]), float(p[3]), 0, 0]], dtype=np.float32),
                                 np.array([[[int(p[4]), int(p[5])]]], dtype=np.int32))
            elif p[0] == "SEARCH":
                items = [tuple(int(t) for t in s.split("/")) for s in p[5:]]
                searches.append(dict(q=p[1], L=int(p[2]), E=int(p[3]), S=int(p[4]),
                                     ids=[a for a, _, _ in items], phi=[b for _, b, _ in items],
                                     d=[c for _, _, c in items]))
            elif p[0] in ("BOA", "WARM"):
                items = [tuple(int(t) for t in s.split("/")) for s in p[8:]]
                (boas if p[0] == "BOA" else warms).append(dict(q=p[1], k=int(p[2]), eps=float(p[3]),
                                 widths=[int(w) for w in p[4].split(",")], final_L=int(p[5]),
                                 E=int(p[6]), S=int(p[7]), ids=[a for a, _ in items],
                                 d=[b for _, b in items]))
    n = len(pts)
    x = np.zeros((n, 4), dtype=np.float32)
    a = np.zeros((n, 1), dtype=np.int32)
    for i, (px, py, av) in pts.items():
        x[i, :2] = (px, py)
        a[i, 0] = av
    A = np.array([adj[i] for i in range(n)], dtype=np.uint32)
    return x, a, A, entry, queries, searches, boas, warms
