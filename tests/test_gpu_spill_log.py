"""GPU parity of the visited set's HBM spill path on an index large enough
for the spill bitmap to keep a log of the ids it holds (a query clears only
their words before it first spills; a full log, or a header in an unknown
state, clears the whole bitmap instead).

Searches repeat on one index, mixing table sizes that spill a little (the
log covers every set bit) and a lot (the log fills up), so that each wave
slot's bitmap passes from query to query and from search to search in both
states. Every result is compared with the oracle exactly: ids, distances,
final widths and per-query expansion and scored counts.
"""
import numpy as np
import pytest

import oracle
from helpers import PAD, random_queries

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def random_graph(n, R, seed):
    """Rows of R - 1 distinct random neighbours (repeats padded) and i + 1
    in the last slot: strongly connected, cheap at any n."""
    rng = np.random.default_rng(seed)
    i = np.arange(n, dtype=np.int64)[:, None]
    rows = np.sort((i + rng.integers(1, n, size=(n, R - 1))) % n, axis=1).astype(np.uint32)
    rows[:, 1:][rows[:, 1:] == rows[:, :-1]] = PAD
    adj = np.empty((n, R), dtype=np.uint32)
    adj[:, :R - 1] = rows
    nxt = ((i[:, 0] + 1) % n).astype(np.uint32)
    adj[:, R - 1] = np.where((rows == nxt[:, None]).any(1), PAD, nxt)
    return adj


@pytest.fixture(scope="module")
def big():
    import paper_2609_16175_amd as boa
    n, d, m, R = 120_000, 16, 2, 12
    rng = np.random.default_rng(77)
    x = rng.integers(0, 256, size=(n, d)).astype(np.uint8)
    a = rng.integers(0, 100, size=(n, m)).astype(np.int32)
    t = np.zeros(m, dtype=np.int32)
    adj = random_graph(n, R, 77)
    orc = oracle.Index(x, a, t, adj, 5)
    gpu = boa.Index(x, a, t, adj, 5)
    q, r = random_queries(orc, 160, 60, seed=78)
    yield dict(orc=orc, gpu=gpu, q=q, r=r)
    gpu.close()


def gpu_search(ix, q, r, **kw):
    dev = torch.device("cuda:0")
    out = ix.search(torch.from_numpy(q).to(dev), torch.from_numpy(r).to(dev), counters=True, **kw)
    torch.cuda.synchronize()
    return (out.ids.cpu().numpy().view(np.uint32), out.dists.cpu().numpy(), out.final_L.cpu().numpy(),
            out.expansions.cpu().numpy().astype(np.int64), out.scored.cpu().numpy().astype(np.int64))


def assert_parity(got, ref, what):
    ids, dists, fl, E, S = got
    bad = np.flatnonzero((ids != ref.ids).any(1) | (dists != ref.dists).any(1) | (fl != ref.final_L)
                         | (E != ref.expansions) | (S != ref.scored))
    assert bad.size == 0, (f"{what}: {bad.size} queries differ; first {bad[0]}: gpu {ids[bad[0]]} L {fl[bad[0]]} "
                           f"E {E[bad[0]]} S {S[bad[0]]}; oracle {ref.ids[bad[0]]} L {ref.final_L[bad[0]]} "
                           f"E {ref.expansions[bad[0]]} S {ref.scored[bad[0]]}")


def test_spill_log_across_queries_and_searches(big):
    q, r = big["q"], big["r"]
    sched = oracle.schedule(16, 2.0, 256)
    ref = oracle.boa(big["orc"], q, r, 10, sched, eps=0.05)
    ref_warm = oracle.boa_warm(big["orc"], q, r, 10, sched, eps=0.05)
    spilled = 0
    for rep in range(2):
        for slots in (4096, 1024, 2048, 8192):
            for mode, kw in (("phased", {}), ("fused", {"fused": True}), ("split", {"split": True}),
                             ("warm", {"fused": True, "warm": True})):
                got = gpu_search(big["gpu"], q, r, k=10, L0=16, Lmax=256, eps=0.05, lds_hash_slots=slots, **kw)
                assert_parity(got, ref_warm if mode == "warm" else ref, f"{mode} table {slots} repeat {rep}")
                spilled += big["gpu"].stats()["spilled_queries"]
    assert spilled > 0   # the spill path ran


def test_spill_log_fixed_widths(big):
    q, r = big["q"], big["r"]
    for L in (64, 512):
        ref = oracle.boa(big["orc"], q, r, 10, [L])
        for slots in (128, 4096):
            got = gpu_search(big["gpu"], q, r, k=10, fixed_L=L, lds_hash_slots=slots)
            assert_parity(got, ref, f"fixed L={L} table {slots}")


def _table_hash(v, B):
    """The visited table's id mix (a bijection on B <= 24 bits), for
    building inputs: two multiplications by odd 24-bit constants around an
    xor-shift."""
    mask = np.uint64((1 << B) - 1)
    h = (v.astype(np.uint64) * np.uint64(0x3779B1)) & mask
    h ^= h >> np.uint64((B + 1) >> 1)
    return (h * np.uint64(0xEBCA6B)) & mask


def test_ids_without_an_alternate_bucket():
    """Ids of B = 19 bits in a 128-slot table keep 15 bits, and those whose
    15 bits are all ones have no alternate bucket (that entry would read as
    a free slot). The entry's row and theirs link them to each other, so
    each is entered early, met again and, once its bucket fills, spilled;
    results must equal the oracle's."""
    import paper_2609_16175_amd as boa
    n, d, m, R = 300_000, 16, 1, 12
    hv = _table_hash(np.arange(n, dtype=np.uint64), 19)
    special = np.flatnonzero((hv & np.uint64(0x7FFF)) == np.uint64(0x7FFF)).astype(np.uint32)
    assert len(special) >= 4
    adj = random_graph(n, R, 91)
    entry = int(special[0])
    for i, s in enumerate(special):
        others = np.roll(special, -i)[1:R]
        row = adj[s]
        row[len(others):][np.isin(row[len(others):], special)] = PAD   # no repeats in the row
        row[:len(others)] = others
    rng = np.random.default_rng(91)
    x = rng.integers(0, 256, size=(n, d)).astype(np.uint8)
    a = rng.integers(0, 100, size=(n, m)).astype(np.int32)
    t = np.zeros(m, dtype=np.int32)
    orc = oracle.Index(x, a, t, adj, entry)
    gpu = boa.Index(x, a, t, adj, entry)
    q, r = random_queries(orc, 64, 70, seed=92)
    for L in (16, 200):
        ref = oracle.boa(orc, q, r, 10, [L])
        for slots in (128, 256):
            for kw in ({}, {"fused": True}):
                got = gpu_search(gpu, q, r, k=10, fixed_L=L, lds_hash_slots=slots, **kw)
                assert_parity(got, ref, f"special ids L={L} table {slots} {kw}")
    gpu.close()
