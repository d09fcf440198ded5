"""The allocation-free search (boa_search_noalloc) against boa_search.

Both entry points run the same kernels; the allocation-free one works in
the library's static per-GPU scratch array instead of memory it allocates.
Its results must equal boa_search's exactly (ids, distances, final widths,
expansion and scored counts), on two calls in a row with the second one
smaller (the scratch keeps the previous call's contents), and where the
spill bitmaps of the planned grid do not fit the scratch (1M points: the
persistent grid is made smaller).
"""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _boa():
    import paper_2609_16175_amd as boa
    return boa


def _run(ix, q, r, **kw):
    dev = torch.device("cuda:0")
    out = ix.search(torch.from_numpy(q).to(dev), torch.from_numpy(r).to(dev), counters=True, **kw)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (out.ids, out.dists, out.final_L, out.expansions, out.scored)]


def _same(a, b, what):
    for name, x, y in zip(("ids", "dists", "final_L", "expansions", "scored"), a, b):
        assert np.array_equal(x, y), f"{what}: {name} differ"


@pytest.fixture(scope="module")
def tiny():
    from workloads import gen, graph
    wl = gen.TINY
    data = gen.generate(wl)
    adj, entry = graph.build_graph(data.vectors, wl.R, "cpu")
    types = np.array(wl.attr_dtypes, dtype=np.int32)
    ix = _boa().Index(data.vectors, data.attrs, types, adj, entry)
    yield wl, data, ix
    ix.close()


@pytest.mark.parametrize("mode", [{}, {"fused": True}, {"split": True}])
def test_noalloc_equals_search_twice_smaller_second(tiny, mode):
    wl, d, ix = tiny
    kw = dict(k=wl.k, L0=wl.L0, Lmax=wl.Lmax, **mode)
    for sl in (slice(0, 100), slice(50, 87)):   # the second call is smaller
        q, r = d.queries[sl], d.ranges[sl]
        ref = _run(ix, q, r, **kw)
        got = _run(ix, q, r, no_alloc=True, **kw)
        _same(got, ref, f"tiny {mode or 'phased'} queries {sl}")


def test_noalloc_grid_capped_to_scratch():
    """1M points: n/8 = 125 KB of spill bitmap per resident wave, so the
    64 MiB scratch holds fewer wave slots than the planned grid; a forced
    512-slot LDS table makes queries spill into those bitmaps."""
    boa = _boa()
    rng = np.random.default_rng(5)
    n, dim, R = 1_000_000, 16, 8
    x = rng.standard_normal((n, dim), dtype=np.float32)
    attrs = rng.integers(0, 100, size=(n, 1)).astype(np.int32)
    adj = rng.integers(0, n, size=(n, R)).astype(np.uint32)
    adj[:, 0] = (np.arange(n) + 1) % n                         # a ring: every point reachable
    adj[adj == np.arange(n, dtype=np.uint32)[:, None]] = 0xFFFFFFFF   # no self edges
    for j in range(1, R):                                      # no repeated id in a row
        dup = (adj[:, j:j + 1] == adj[:, :j]).any(1)
        adj[dup, j] = 0xFFFFFFFF
    ix = boa.Index(x, attrs, np.zeros(1, np.int32), adj, 0)
    for nq in (600, 250):
        q = rng.standard_normal((nq, dim), dtype=np.float32)
        lo = rng.integers(0, 50, size=nq)
        r = np.stack([lo, lo + 49], axis=1).astype(np.int32)[:, None, :]
        for mode in ({}, {"fused": True}, {"split": True}):
            kw = dict(k=10, schedule=[16, 64], eps=0.05, lds_hash_slots=512, **mode)
            ref = _run(ix, q, r, **kw)
            got = _run(ix, q, r, no_alloc=True, **kw)
            _same(got, ref, f"1M points nq={nq} {mode or 'phased'}")
    ix.close()


def test_noalloc_rejects_what_it_cannot_run(tiny):
    boa = _boa()
    wl, d, ix = tiny
    dev = torch.device("cuda:0")
    q = torch.from_numpy(d.queries[:4]).to(dev)
    r = torch.from_numpy(d.ranges[:4]).to(dev)
    with pytest.raises(boa.BoaError) as e:
        ix.search(q, r, k=wl.k, boa_plus=True, no_alloc=True)
    assert e.value.code == -4
    # more queries than the scratch is sized for: refused before any device
    # work (the buffers are never touched, so small ones suffice)
    ids = torch.empty((4, wl.k), dtype=torch.int32, device=dev)
    dists = torch.empty((4, wl.k), dtype=torch.float32, device=dev)
    fl = torch.empty((4,), dtype=torch.int32, device=dev)
    p = boa.default_params()
    rc = boa.lib().boa_search_noalloc(ix._h, q.data_ptr(), r.data_ptr(), (1 << 18) + 1, C.byref(p),
                                      ids.data_ptr(), dists.data_ptr(), fl.data_ptr(), None, None,
                                      torch.cuda.current_stream(dev).cuda_stream)
    assert rc == -1 and b"maximum" in boa.lib().boa_last_error()
