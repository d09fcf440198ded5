"""GPU parity of the product-quantised traversal with exact re-rank (Alg. 2
"PQDist"; Sec. III-B steps 2, 6 and 8) against the oracle's mirror mode:
ids, distances, final widths and per-query expansion and scored counts
identical, in every driver mode, at table sizes that span the kernel's
variants (16 to 256 subspaces), for float32 and uint8 vectors.
"""
import numpy as np
import pytest

import oracle
from helpers import PAD, random_arrays, random_queries
from workloads import pq

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _boa():
    import paper_2609_16175_amd as boa
    return boa


def gpu_search(ix, q, r, **kw):
    dev = torch.device("cuda:0")
    out = ix.search(torch.from_numpy(np.ascontiguousarray(q)).to(dev),
                    torch.from_numpy(np.ascontiguousarray(r, dtype=np.int32)).to(dev), counters=True, **kw)
    torch.cuda.synchronize()
    return (out.ids.cpu().numpy().view(np.uint32), out.dists.cpu().numpy(), out.final_L.cpu().numpy(),
            out.expansions.cpu().numpy().astype(np.int64), out.scored.cpu().numpy().astype(np.int64))


def assert_parity(got, ref, what=""):
    ids, dists, fl, E, S = got
    bad = np.flatnonzero((ids != ref.ids).any(1) | (dists != ref.dists).any(1) | (fl != ref.final_L)
                         | (E != ref.expansions) | (S != ref.scored))
    if bad.size:
        i = bad[0]
        raise AssertionError(f"{what}: {bad.size} queries differ; first {i}: gpu {ids[i]} {dists[i]} L {fl[i]} "
                             f"E {E[i]} S {S[i]}; oracle {ref.ids[i]} {ref.dists[i]} L {ref.final_L[i]} "
                             f"E {ref.expansions[i]} S {ref.scored[i]}")


@pytest.fixture(scope="module")
def tiny():
    from workloads import gen, graph
    wl = gen.TINY
    d = gen.generate(wl)
    adj, entry = graph.build_graph(d.vectors, wl.R, "cpu")
    types = np.array(wl.attr_dtypes, dtype=np.int32)
    cb = pq.train(d.vectors, 8, seed=1)
    codes = pq.encode(d.vectors, cb)
    orc = oracle.Index(d.vectors, d.attrs, types, adj, entry, cb, codes)
    gpu = _boa().Index(d.vectors, d.attrs, types, adj, entry)
    gpu.set_pq(cb, codes)
    yield dict(wl=wl, d=d, orc=orc, gpu=gpu)
    gpu.close()


MODES = {"phased": {}, "fused": {"fused": True}, "split": {"split": True},
         "boa_plus": {"boa_plus": True, "sub_batches": 3}}


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("eps", [0.0, 0.05, 0.2])
def test_tiny_pq(tiny, mode, eps):
    wl, d = tiny["wl"], tiny["d"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, sched, eps=eps)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, eps=eps, pq=True,
                     **MODES[mode])
    assert_parity(got, ref, f"tiny pq {mode} eps={eps}")


def test_tiny_pq_warm_and_fixed(tiny):
    wl, d = tiny["wl"], tiny["d"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa_warm(tiny["orc"], d.queries, d.ranges, wl.k, sched, eps=0.02)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, eps=0.02, pq=True,
                     fused=True, warm=True)
    assert_parity(got, ref, "tiny pq warm")
    for L in (10, 64, 300):
        ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, [L])
        got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, fixed_L=L, pq=True)
        assert_parity(got, ref, f"tiny pq fixed L={L}")
    # a forced small visited table (spills to the HBM bitmap)
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, sched)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, pq=True, lds_hash_slots=64)
    assert_parity(got, ref, "tiny pq spill")


SHAPES = [
    # dtype, d, M, m, R, f32 column
    ("f32", 32, 16, 2, 17, True),
    ("f32", 96, 24, 3, 64, True),
    ("f32", 128, 64, 2, 33, False),
    ("f32", 768, 192, 4, 48, True),
    ("f32", 1024, 256, 1, 12, False),
    ("u8", 16, 4, 1, 9, False),
    ("u8", 128, 32, 2, 32, False),
    ("u8", 96, 48, 5, 40, True),
]


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{s[0]}-d{s[1]}-M{s[2]}-m{s[3]}-R{s[4]}" for s in SHAPES])
def test_shapes_pq(shape):
    dtype, d, M, m, R, f32col = shape
    x, a, t, adj, e = random_arrays(n=3000, d=d, m=m, R=R, dtype=dtype, seed=d + M, f32_col=f32col)
    cb = pq.train(x, M, seed=M, iters=6)
    codes = pq.encode(x, cb)
    orc = oracle.Index(x, a, t, adj, e, cb, codes)
    gpu = _boa().Index(x, a, t, adj, e)
    gpu.set_pq(cb, codes)
    q, r = random_queries(orc, 150, 40, seed=d + 7, f32_col=f32col)
    sched = oracle.schedule(16, 2.0, 256)
    ref = oracle.boa(orc, q, r, 10, sched, eps=0.1)
    for mode in ({}, {"fused": True}, {"split": True}):
        got = gpu_search(gpu, q, r, k=10, L0=16, Lmax=256, eps=0.1, pq=True, **mode)
        assert_parity(got, ref, f"shape {shape} {mode or 'phased'}")
    ref = oracle.boa_warm(orc, q, r, 10, [10, 100, 200], eps=0.05)
    got = gpu_search(gpu, q, r, k=10, schedule=[10, 100, 200], eps=0.05, pq=True, fused=True, warm=True)
    assert_parity(got, ref, f"shape {shape} warm")
    gpu.close()


def test_exact_codebook_equals_the_exact_search():
    """Integer data whose subvectors are exactly the codebook's centroids:
    the asymmetric distance is the exact distance, so the PQ search returns
    what the exact search returns, with the same counts."""
    rng = np.random.default_rng(3)
    n, d, M = 3000, 32, 8
    patterns = rng.integers(0, 9, size=(M, 16, 4))
    c = rng.integers(0, 16, size=(n, M))
    x = np.concatenate([patterns[j][c[:, j]] for j in range(M)], axis=1).astype(np.float32)
    _, a, t, adj, e = random_arrays(n=n, d=d, m=2, R=12, seed=3, f32_col=True)
    gpu = _boa().Index(x, a, t, adj, e)
    gpu.set_pq(patterns.astype(np.float32), (c[:, 0::2] | (c[:, 1::2] << 4)).astype(np.uint8))
    q = rng.integers(0, 9, size=(100, d)).astype(np.float32)
    _, r = random_queries(oracle.Index(x, a, t, adj, e), 100, 40, seed=3, f32_col=True)
    exact = gpu_search(gpu, q, r, k=10, L0=16, Lmax=128, eps=0.05)
    withpq = gpu_search(gpu, q, r, k=10, L0=16, Lmax=128, eps=0.05, pq=True)
    for u, v in zip(exact, withpq):
        np.testing.assert_array_equal(u, v)
    gpu.close()


def test_pq_needs_codes(tiny):
    boa = _boa()
    from workloads import gen, graph
    d = tiny["d"]
    types = np.array(tiny["wl"].attr_dtypes, dtype=np.int32)
    plain = boa.Index(d.vectors, d.attrs, types, graph.build_graph(d.vectors, 16, "cpu")[0], 0)
    q = torch.from_numpy(d.queries[:4]).to("cuda:0")
    r = torch.from_numpy(d.ranges[:4]).to("cuda:0")
    with pytest.raises(boa.BoaError) as ex:
        plain.search(q, r, k=10, pq=True)
    assert ex.value.code == -1
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=200, L0=256, Lmax=512, pq=True)   # k above 128
    with pytest.raises(boa.BoaError) as ex:   # M odd and not dividing d: refused by the library
        plain.set_pq(np.zeros((3, 16, 10), np.float32), np.zeros((d.vectors.shape[0], 1), np.uint8))
    assert ex.value.code == -1
    plain.close()
