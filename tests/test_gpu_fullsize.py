"""GPU parity at the workloads' full sizes, in the benchmark's launch
configuration: the whole 10,000-query batch runs on the GPU (fused, split, phased
and BOA+ modes, and the fixed-width baseline); a seeded sample of queries is
recomputed by the CPU oracle one by one and compared row by row. Because a
query's result does not depend on the rest of the batch (every phase
restarts the search), the oracle's sample is an exact check of those rows.
"""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SAMPLE = 200
SAMPLE_FIXED = 48


def _setup(name):
    import paper_2609_16175_amd as boa
    from workloads import gen, graph
    wl = gen.BY_NAME[name]
    data = gen.generate(wl)
    types = np.array(wl.attr_dtypes, dtype=np.int32)
    # the benchmark's graph: vector edges plus attribute-aware edges (from
    # k-means lists above 2M points: about 4 minutes for u8-10M-d128)
    adj, entry = graph.build_graph(data.vectors, wl.R, device="cuda:0", attrs=data.attrs, attr_dtypes=types)
    torch.cuda.empty_cache()
    gpu = boa.Index(data.vectors, data.attrs, types, adj, entry)
    orc = oracle.Index(data.vectors, data.attrs, types, adj, entry)
    q = torch.from_numpy(data.queries).to("cuda:0")
    r = torch.from_numpy(data.ranges).to("cuda:0")
    sample = np.sort(np.random.default_rng(7).choice(wl.nq, SAMPLE, replace=False))
    return dict(wl=wl, data=data, gpu=gpu, orc=orc, q=q, r=r, sample=sample, adj=adj, entry=entry)


def _rows(out, sel):
    ids = out.ids.cpu().numpy().view(np.uint32)[sel]
    return (ids, out.dists.cpu().numpy()[sel], out.final_L.cpu().numpy()[sel],
            out.expansions.cpu().numpy().astype(np.int64)[sel], out.scored.cpu().numpy().astype(np.int64)[sel])


def _check(got, ref, what):
    ids, dists, fl, E, S = got
    bad = np.flatnonzero((ids != ref.ids).any(1) | (dists != ref.dists).any(1) | (fl != ref.final_L)
                         | (E != ref.expansions) | (S != ref.scored))
    assert bad.size == 0, (f"{what}: {bad.size} sampled queries differ; first row {bad[0]}: "
                           f"gpu {ids[bad[0]]} / {dists[bad[0]]} L {fl[bad[0]]}; "
                           f"oracle {ref.ids[bad[0]]} / {ref.dists[bad[0]]} L {ref.final_L[bad[0]]}")


@pytest.fixture(scope="module",
                params=["sift-like-1M-d128", "deep-like-1M-d96", "dblp-like-1M-d768", "u8-10M-d128"])
def full(request):
    env = _setup(request.param)
    yield env
    env["gpu"].close()


def test_full_size_index_builds(full):
    """Graph construction is its own test item (minutes at 10M points): the
    adjacency is well formed and every point is reachable from the entry."""
    from workloads import graph
    wl = full["wl"]
    adj = full["adj"]
    assert adj.shape == (wl.n, wl.R)
    assert graph._reachable(wl.n, adj, full["entry"]).all()


def test_full_size_adaptive_sampled(full):
    wl, d, s = full["wl"], full["data"], full["sample"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(full["orc"], d.queries[s], d.ranges[s], wl.k, sched, threads=16)
    for mode in ({"fused": True}, {"split": True}, {}, {"boa_plus": True, "sub_batches": wl.sub_batches}):
        out = full["gpu"].search(full["q"], full["r"], k=wl.k, L0=wl.L0, Lmax=wl.Lmax, counters=True, **mode)
        torch.cuda.synchronize()
        _check(_rows(out, s), ref, f"{wl.name} {mode or 'phased'}")
        # every result id satisfies the predicates of its query (whole batch)
        ids = out.ids.cpu().numpy().view(np.uint32)
        assert ids.shape == (wl.nq, wl.k)


def test_full_size_fixed_width_sampled(full):
    wl, d = full["wl"], full["data"]
    s = full["sample"][:SAMPLE_FIXED]
    ref = oracle.boa(full["orc"], d.queries[s], d.ranges[s], wl.k, [500], threads=16)
    out = full["gpu"].search(full["q"], full["r"], k=wl.k, fixed_L=500, counters=True)
    torch.cuda.synchronize()
    _check(_rows(out, s), ref, f"{wl.name} fixed L=500")
