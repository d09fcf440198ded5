"""Pins of the oracle's product-quantised traversal (Alg. 2 "PQDist";
Sec. III-B: per-query distance tables, asymmetric distances, exact re-rank
of the accumulated candidates at convergence).

Each check compares the oracle with something other than itself: float64
numpy, the squared distance to the decoded vector (the identity that
defines an asymmetric distance), the exact search (which PQ must equal
when the codebook reproduces the data exactly), and exhaustive search
(which PQ at full width must equal after the exact re-rank).
"""
import numpy as np
import pytest

import oracle
from helpers import PAD, numpy_valid, random_arrays, random_queries
from workloads import pq


def _rand_pq(n=400, d=16, M=4, seed=0, dtype="f32"):
    x, a, t, adj, e = random_arrays(n=n, d=d, m=2, R=10, dtype=dtype, seed=seed, f32_col=True)
    cb = pq.train(x, M, seed=seed, iters=6)
    codes = pq.encode(x, cb)
    return oracle.Index(x, a, t, adj, e, cb, codes)


@pytest.mark.parametrize("d,M", [(16, 4), (32, 16), (96, 24), (128, 32)])
def test_table_is_the_squared_subvector_distance(d, M):
    ix = _rand_pq(d=d, M=M, seed=d)
    ds = d // M
    rng = np.random.default_rng(d)
    for _ in range(5):
        q = rng.normal(size=d).astype(np.float32)
        t = oracle.pq_table(ix, q)
        ref = ((q.astype(np.float64).reshape(M, 1, ds) - ix.pq_codebook.astype(np.float64)) ** 2).sum(-1)
        np.testing.assert_allclose(t, ref, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("d,M", [(16, 4), (32, 16), (96, 24), (128, 32), (768, 192)])
def test_asymmetric_distance_is_the_distance_to_the_decoded_vector(d, M):
    ix = _rand_pq(n=300, d=d, M=M, seed=d + 1)
    rng = np.random.default_rng(d + 1)
    dec = pq.decode(ix.pq_codes, ix.pq_codebook)
    for _ in range(3):
        q = rng.normal(size=d).astype(np.float32)
        t = oracle.pq_table(ix, q)
        for v in rng.integers(0, ix.n, 20):
            got = oracle.pq_dist(t, ix.pq_codes[v])
            ref = ((dec[v] - q.astype(np.float64)) ** 2).sum()
            assert abs(got - ref) <= 1e-5 * ref + 1e-6


def test_every_subspace_and_nibble_counts():
    ix = _rand_pq(d=32, M=16, seed=5)
    q = np.random.default_rng(5).normal(size=32).astype(np.float32)
    t = oracle.pq_table(ix, q).astype(np.float64)
    code = ix.pq_codes[7].copy()
    base = oracle.pq_dist(t.astype(np.float32), code)
    c = pq.unpack(code[None])[0]
    for m in range(16):
        new = (int(c[m]) + 5) % 16
        code2 = code.copy()
        code2[m // 2] = (code2[m // 2] & (0xF0 if m % 2 == 0 else 0x0F)) | (new << (4 * (m % 2)))
        got = oracle.pq_dist(t.astype(np.float32), code2)
        assert abs((got - base) - (t[m, new] - t[m, c[m]])) <= 1e-4 * max(1.0, abs(base))


def _exact_codebook_index(seed, dtype):
    """Integer data whose every 4-dim subvector is one of 16 patterns, and
    a codebook holding exactly those: decoding reproduces the data, and
    every sum involved is an exact integer, so the asymmetric distance
    equals the exact distance bit for bit."""
    rng = np.random.default_rng(seed)
    n, d, M = 600, 32, 8
    patterns = rng.integers(0, 9, size=(M, 16, 4))
    c = rng.integers(0, 16, size=(n, M))
    x = np.concatenate([patterns[m][c[:, m]] for m in range(M)], axis=1)
    x = x.astype(np.uint8 if dtype == "u8" else np.float32)
    _, a, t, _, e = random_arrays(n=n, d=d, m=2, R=10, seed=seed, f32_col=True)
    from helpers import ring_knn_graph
    adj = ring_knn_graph(x.astype(np.float32) + 1e-3 * rng.normal(size=x.shape).astype(np.float32), 10, seed)
    cb = patterns.astype(np.float32)
    codes = (c[:, 0::2] | (c[:, 1::2] << 4)).astype(np.uint8)
    return x, a, t, adj, e, cb, codes


@pytest.mark.parametrize("dtype", ["f32", "u8"])
def test_exact_codebook_gives_the_exact_search(dtype):
    x, a, t, adj, e, cb, codes = _exact_codebook_index(11, dtype)
    plain = oracle.Index(x, a, t, adj, e)
    withpq = oracle.Index(x, a, t, adj, e, cb, codes)
    assert np.array_equal(pq.decode(codes, cb), x.astype(np.float64))
    rng = np.random.default_rng(12)
    q = rng.integers(0, 9, size=(40, 32)).astype(x.dtype)
    _, r = random_queries(plain, 40, 40, seed=12, f32_col=True)
    for sched in ([16, 32, 64], [10]):
        a1 = oracle.boa(plain, q, r, 10, sched, eps=0.1)
        a2 = oracle.boa(withpq, q, r, 10, sched, eps=0.1)
        for f in ("ids", "dists", "final_L", "expansions", "scored"):
            np.testing.assert_array_equal(getattr(a1, f), getattr(a2, f))
    w1 = oracle.boa_warm(plain, q, r, 10, [16, 32, 64], eps=0.1)
    w2 = oracle.boa_warm(withpq, q, r, 10, [16, 32, 64], eps=0.1)
    np.testing.assert_array_equal(w1.ids, w2.ids)
    np.testing.assert_array_equal(w1.scored, w2.scored)


@pytest.mark.parametrize("dtype", ["f32", "u8"])
def test_full_width_pq_search_reranks_to_the_exact_answer(dtype):
    """At a width of at least n nothing is cut: every reachable point is
    scored and the valid ones are all in the final list, so the exact
    re-rank returns the exact filtered top-k (Def. 1)."""
    ix = _rand_pq(n=300, d=16, M=4, seed=21, dtype=dtype)
    q, r = random_queries(ix, 15, 40, seed=21, f32_col=True)
    res = oracle.boa(ix, q, r, 10, [ix.n])
    bi, bd, nv = oracle.bruteforce(ix, q, r, 10)
    np.testing.assert_array_equal(res.ids, bi)
    np.testing.assert_array_equal(res.dists, bd)
    assert (res.scored == ix.n).all()


def test_pq_result_invariants():
    """Narrow widths: returned ids satisfy the predicates, the reported
    distances are exact distances, rows ascend by (exact distance, id)."""
    ix = _rand_pq(n=1500, d=32, M=8, seed=31)
    q, r = random_queries(ix, 50, 30, seed=31, f32_col=True)
    for run in (lambda: oracle.boa(ix, q, r, 10, [16, 32, 64], eps=0.05),
                lambda: oracle.boa_warm(ix, q, r, 10, [16, 32, 64], eps=0.05)):
        res = run()
        for i in range(q.shape[0]):
            got = res.ids[i][res.ids[i] != PAD]
            assert numpy_valid(ix, r[i])[got.astype(np.int64)].all()
            dd = res.dists[i][:len(got)]
            for j, g in enumerate(got):
                assert dd[j] == oracle.dist(ix.vectors[g], q[i])
            assert list(zip(dd, got)) == sorted(zip(dd, got))
    # the traversal's worklist orders by asymmetric distance
    ids, ph, d, ln, E, S = oracle.search_lists(ix, q[:5], r[:5], 16)
    for i in range(5):
        t = oracle.pq_table(ix, q[i])
        for j in range(ln[i]):
            assert d[i, j] == oracle.pq_dist(t, ix.pq_codes[ids[i, j]])
