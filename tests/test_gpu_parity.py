"""GPU parity: the HIP search (through the C ABI) against the CPU oracle.

Bar: ids, distances, final widths and per-query expansion/scored counts
identical to the oracle (both sides use one float32 summation order and
take every decision in the same precision), on seeded inputs spanning
several wave rounds, ragged candidate counts and the edge cases.
"""
import numpy as np
import pytest

import oracle
from helpers import PAD, random_arrays, random_queries

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _boa():
    import paper_2609_16175_amd as boa
    return boa


def gpu_search(ix, q, r, **kw):
    dev = torch.device("cuda:0")
    qt = torch.from_numpy(np.ascontiguousarray(q)).to(dev)
    rt = torch.from_numpy(np.ascontiguousarray(r, dtype=np.int32)).to(dev)
    out = ix.search(qt, rt, counters=True, **kw)
    torch.cuda.synchronize()
    return (out.ids.cpu().numpy().view(np.uint32), out.dists.cpu().numpy(), out.final_L.cpu().numpy(),
            out.expansions.cpu().numpy().astype(np.int64), out.scored.cpu().numpy().astype(np.int64))


def assert_parity(got, ref, what=""):
    ids, dists, fl, E, S = got
    bad = np.flatnonzero((ids != ref.ids).any(1) | (dists != ref.dists).any(1) | (fl != ref.final_L)
                         | (E != ref.expansions) | (S != ref.scored))
    if bad.size:
        i = bad[0]
        raise AssertionError(
            f"{what}: {bad.size} queries differ; first {i}: gpu ids {ids[i]} oracle {ref.ids[i]}; "
            f"gpu d {dists[i]} oracle {ref.dists[i]}; L {fl[i]} vs {ref.final_L[i]}; "
            f"E {E[i]} vs {ref.expansions[i]}; S {S[i]} vs {ref.scored[i]}")


# ---------------------------------------------------------------------------
# the tiny workload: 10k points, d=32, R=16, m=1, 100 queries, L 16 -> 128

@pytest.fixture(scope="module")
def tiny():
    from workloads import gen, graph
    wl = gen.TINY
    data = gen.generate(wl)
    adj, entry = graph.build_graph(data.vectors, wl.R, "cpu")
    types = np.array(wl.attr_dtypes, dtype=np.int32)
    boa = _boa()
    return dict(wl=wl, data=data, orc=oracle.Index(data.vectors, data.attrs, types, adj, entry),
                gpu=boa.Index(data.vectors, data.attrs, types, adj, entry))


MODES = {"phased": {}, "fused": {"fused": True}, "split": {"split": True}}


@pytest.mark.parametrize("mode", list(MODES))
def test_tiny_adaptive(tiny, mode):
    wl, d = tiny["wl"], tiny["data"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, sched)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, **MODES[mode])
    assert_parity(got, ref, f"tiny adaptive {mode}")
    st = tiny["gpu"].stats()
    assert [p["L"] for p in st["phases"]] == sched
    for p, rp in zip(st["phases"], ref.phases):
        assert (p["active"], p["confident"], p["expansions"], p["scored"]) == \
            (rp["active"], rp["confident"], rp["expansions"], rp["scored"])


@pytest.mark.parametrize("sub", [1, 3, 10, 100])
def test_tiny_boa_plus(tiny, sub):
    """BOA+ (sub-batched first phase, pooled escalation on a second stream)
    settles every query exactly as BOA does (Sec. III-A)."""
    wl, d = tiny["wl"], tiny["data"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, sched, eps=0.02)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, eps=0.02,
                     boa_plus=True, sub_batches=sub)
    assert_parity(got, ref, f"BOA+ sub_batches={sub}")
    st = tiny["gpu"].stats()
    for p, rp in zip(st["phases"], ref.phases):
        assert (p["active"], p["confident"], p["expansions"], p["scored"]) == \
            (rp["active"], rp["confident"], rp["expansions"], rp["scored"])
    assert st["phases"][0]["launches"] == min(sub, d.queries.shape[0])


@pytest.mark.parametrize("L", [10, 16, 64, 128, 500])
def test_tiny_fixed_width(tiny, L):
    wl, d = tiny["wl"], tiny["data"]
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, [L])
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, fixed_L=L)
    assert_parity(got, ref, f"tiny fixed L={L}")


@pytest.mark.parametrize("slots,mode", [(64, "phased"), (256, "phased"), (64, "fused"), (64, "split")])
def test_forced_spill_changes_nothing(tiny, slots, mode):
    """A tiny LDS visited table sends almost every insert to the HBM bitmap."""
    wl, d = tiny["wl"], tiny["data"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, sched)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax,
                     lds_hash_slots=slots, **MODES[mode])
    assert_parity(got, ref, f"spill slots={slots}")
    assert tiny["gpu"].stats()["spilled_queries"] > 0
    # and twice in a row: a wave slot's bitmap is reset by the next query that spills
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax,
                     lds_hash_slots=slots, **MODES[mode])
    assert_parity(got, ref, f"spill slots={slots}, repeated")


@pytest.mark.parametrize("eps", [0.0, 0.005, 0.05])
def test_split_escalation_bitmap_and_table(tiny, eps):
    """The split search's escalation launch keeps its visited set as an LDS
    bitmap over all ids when that fits (10k points: 1.25 KB) and as the
    hashed table when a table size is forced; both are exact sets, so both
    equal the oracle, with almost every query escalating at small eps."""
    wl, d = tiny["wl"], tiny["data"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, sched, eps=eps)
    assert ref.phases[1]["active"] > 0
    for slots, waves in ((0, 0), (0, 1), (4096, 0)):
        got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, eps=eps,
                         split=True, lds_hash_slots=slots, escalation_waves=waves)
        assert_parity(got, ref, f"split eps={eps} slots={slots} escalation_waves={waves}")


@pytest.mark.parametrize("eps", [0.0, 0.02, 0.05])
def test_split_two_wave_escalation(tiny, eps):
    """The escalation launch with two waves per query (one merging the
    worklist, one expanding the node it expects next and taking the guess
    back when the selection differs) against the oracle and the one-wave
    launch. Widths 10, 20, 40, 80: no query is confident at 10 (it needs
    more than k valid entries), some stop at 20 inside the escalation launch
    (eps 0.02: 27 of 100), the rest run to 80. Twice with two waves."""
    wl, d = tiny["wl"], tiny["data"]
    sched = [10, 20, 40, 80]
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, 10, sched, eps=eps)
    assert ref.phases[1]["active"] == d.queries.shape[0]
    for waves in (0, 1, 0):
        got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=10, schedule=sched, eps=eps,
                         split=True, escalation_waves=waves)
        assert_parity(got, ref, f"split eps={eps} escalation_waves={waves}")
        st = tiny["gpu"].stats()
        for p, rp in zip(st["phases"], ref.phases):
            assert (p["active"], p["confident"], p["expansions"], p["scored"]) == \
                (rp["active"], rp["confident"], rp["expansions"], rp["scored"])
    with pytest.raises(_boa().BoaError):
        gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, split=True, escalation_waves=2)


@pytest.mark.parametrize("mode", list(MODES))
def test_paper_schedule(tiny, mode):
    """The paper's experiments use widths 10, 100, 200 (Sec. IV)."""
    wl, d = tiny["wl"], tiny["data"]
    ref = oracle.boa(tiny["orc"], d.queries, d.ranges, 10, [10, 100, 200], eps=0.02)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=10, schedule=[10, 100, 200], eps=0.02,
                     **MODES[mode])
    assert_parity(got, ref, "schedule 10/100/200")
    st = tiny["gpu"].stats()
    for p, rp in zip(st["phases"], ref.phases):
        assert (p["active"], p["confident"], p["expansions"], p["scored"]) == \
            (rp["active"], rp["confident"], rp["expansions"], rp["scored"])


def test_single_query_equals_batch(tiny):
    wl, d = tiny["wl"], tiny["data"]
    full = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax)
    for i in (0, 37, 99):
        one = gpu_search(tiny["gpu"], d.queries[i:i + 1], d.ranges[i:i + 1], k=wl.k, L0=wl.L0, Lmax=wl.Lmax)
        for a, b in zip(one, full):
            np.testing.assert_array_equal(a[0], b[i])


def test_tau_residual(tiny):
    wl, d = tiny["wl"], tiny["data"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    for tau in (0.01, 0.05, 0.5):
        ref = oracle.boa(tiny["orc"], d.queries, d.ranges, wl.k, sched, eps=0.2, tau=tau)
        got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, eps=0.2, tau=tau)
        assert_parity(got, ref, f"tau={tau}")


def test_k_equal_first_width_and_k_one(tiny):
    wl, d = tiny["wl"], tiny["data"]
    for k, L0 in ((16, 16), (1, 16), (10, 10)):
        sched = oracle.schedule(L0, 2.0, 128)
        ref = oracle.boa(tiny["orc"], d.queries, d.ranges, k, sched)
        got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=k, L0=L0, Lmax=128)
        assert_parity(got, ref, f"k={k} L0={L0}")


def test_empty_valid_sets_and_unbounded(tiny):
    wl, d = tiny["wl"], tiny["data"]
    r = d.ranges.copy()
    r[::3, 0] = [5000, 6000]                      # nothing valid
    r[1::3, 0] = [-2**31, 2**31 - 1]              # everything valid
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(tiny["orc"], d.queries, r, wl.k, sched)
    got = gpu_search(tiny["gpu"], d.queries, r, k=wl.k, L0=wl.L0, Lmax=wl.Lmax)
    assert_parity(got, ref, "empty/unbounded ranges")
    assert (got[0][::3] == PAD).all() and np.isinf(got[1][::3]).all()


def test_no_queries(tiny):
    boa = _boa()
    q = torch.zeros((0, 32), dtype=torch.float32, device="cuda:0")
    r = torch.zeros((0, 1, 2), dtype=torch.int32, device="cuda:0")
    out = tiny["gpu"].search(q, r, k=10)
    assert out.ids.shape == (0, 10)
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=20, L0=16)          # k above the first width
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=10, Lmax=4096)       # beyond the widest supported width
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=10, tau=1.0)
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=10, lds_hash_slots=100)
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=10, tau=0.1, fused=True)
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=10, tau=0.1, boa_plus=True)
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=10, fused=True, boa_plus=True)
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=10, tau=0.1, split=True)
    with pytest.raises(boa.BoaError):
        tiny["gpu"].search(q, r, k=10, split=True, boa_plus=True)
    with pytest.raises(ValueError):
        tiny["gpu"].search(q, r, k=10, split=True, fused=True)


# ---------------------------------------------------------------------------
# shapes: float32 / uint8, dimensions across the kernel variants, m up to 8,
# degrees with ragged wave rounds, float32 attribute columns

SHAPES = [
    # dtype, d, m, R, f32 column
    ("f32", 4, 1, 8, False),
    ("f32", 32, 3, 33, True),
    ("f32", 96, 2, 64, False),
    ("f32", 128, 2, 64, True),
    ("f32", 200, 4, 17, False),
    ("f32", 768, 4, 48, True),
    ("f32", 1024, 8, 12, True),
    ("u8", 16, 1, 9, False),
    ("u8", 128, 2, 32, False),
    ("u8", 96, 5, 40, True),
    ("u8", 1024, 2, 64, False),
]


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{s[0]}-d{s[1]}-m{s[2]}-R{s[3]}" for s in SHAPES])
def test_shapes(shape):
    dtype, d, m, R, f32col = shape
    boa = _boa()
    arrs = random_arrays(n=3000, d=d, m=m, R=R, dtype=dtype, seed=d + m + R, f32_col=f32col)
    orc = oracle.Index(*arrs)
    gpu = boa.Index(*arrs)
    q, r = random_queries(orc, 150, 40, seed=d, f32_col=f32col)
    sched = oracle.schedule(16, 2.0, 256)
    ref = oracle.boa(orc, q, r, 10, sched, eps=0.1)
    got = gpu_search(gpu, q, r, k=10, L0=16, Lmax=256, eps=0.1)
    assert_parity(got, ref, f"shape {shape}")
    got = gpu_search(gpu, q, r, k=10, L0=16, Lmax=256, eps=0.1, fused=True)
    assert_parity(got, ref, f"shape {shape} fused")
    got = gpu_search(gpu, q, r, k=10, L0=16, Lmax=256, eps=0.1, split=True)
    assert_parity(got, ref, f"shape {shape} split")
    got = gpu_search(gpu, q, r, k=10, L0=16, Lmax=256, eps=0.1, boa_plus=True, sub_batches=4)
    assert_parity(got, ref, f"shape {shape} BOA+")
    ref = oracle.boa(orc, q, r, 10, [300])
    got = gpu_search(gpu, q, r, k=10, fixed_L=300, lds_hash_slots=2 * 64 if R < 64 else 256)
    assert_parity(got, ref, f"shape {shape} fixed 300 with spill")
    gpu.close()


# ---------------------------------------------------------------------------
# attribute cells at the edges of their types: float32 zeros of both signs,
# infinities, NaNs (either sign, quiet and signalling), denormals and
# extremes; int32 extremes; bounds of the same kinds, NaN bounds and empty
# ranges. The oracle compares each column in its own type.

def _f32_cells(vals):
    return np.asarray(vals, dtype=np.float32).view(np.int32)


F32_EDGE_CELLS = np.concatenate([
    _f32_cells([0.0, -0.0, np.inf, -np.inf, 1e-45, -1e-45, 1.1754944e-38, -1.1754944e-38,
                3.4028235e38, -3.4028235e38, 1.0, -1.0, 0.5, -0.5]),
    np.array([0x7FC00000, 0x7F800001, 0xFFC00000, 0xFFFFFFFF], dtype=np.uint32).view(np.int32),   # NaNs
])
I32_EDGE_CELLS = np.array([-2**31, -2**31 + 1, -1, 0, 1, 2**31 - 2, 2**31 - 1], dtype=np.int32)


def _edge_case_inputs(dtype, d, R, seed):
    """An index whose columns are (int32, float32, float32): a quarter of the
    cells from the edge sets, the rest ordinary; and queries whose bounds mix
    the same values with ordinary ones (empty and NaN-bounded ranges too)."""
    x, attrs, _, adj, entry = random_arrays(n=3000, d=d, m=3, R=R, dtype=dtype, seed=seed)
    rng = np.random.default_rng(seed + 7)
    n = x.shape[0]
    types = np.array([0, 1, 1], dtype=np.int32)
    a = np.empty((n, 3), dtype=np.int32)
    a[:, 0] = rng.integers(-50, 50, n)
    a[:, 1] = _f32_cells(rng.normal(size=n))
    a[:, 2] = _f32_cells(np.round(rng.normal(size=n), 1))   # many exact zeros, some -0.0
    edge = rng.random((n, 3)) < 0.25
    a[:, 0] = np.where(edge[:, 0], rng.choice(I32_EDGE_CELLS, n), a[:, 0])
    a[:, 1] = np.where(edge[:, 1], rng.choice(F32_EDGE_CELLS, n), a[:, 1])
    a[:, 2] = np.where(edge[:, 2], rng.choice(F32_EDGE_CELLS, n), a[:, 2])
    orc = oracle.Index(x, a, types, adj, entry)
    q, _ = random_queries(orc, 160, 40, seed=seed)
    nq = q.shape[0]
    r = np.empty((nq, 3, 2), dtype=np.int32)
    lo0 = rng.integers(-70, -20, nq)
    r[:, 0, 0], r[:, 0, 1] = lo0, lo0 + rng.integers(-5, 130, nq)          # a few lo > hi
    ii = rng.random(nq) < 0.15
    r[ii, 0, 0] = rng.choice(I32_EDGE_CELLS[:3], ii.sum())
    r[ii, 0, 1] = rng.choice(I32_EDGE_CELLS[3:], ii.sum())
    r[:, 1, 0], r[:, 1, 1] = _f32_cells(-2.5 + rng.random(nq)), _f32_cells(1.5 + rng.random(nq))
    r[:, 2, 0], r[:, 2, 1] = _f32_cells(np.full(nq, -3.0)), _f32_cells(np.full(nq, 3.0))
    for col in (1, 2):
        for side in (0, 1):
            jj = rng.random(nq) < 0.12
            r[jj, col, side] = rng.choice(F32_EDGE_CELLS, jj.sum())
    r[rng.random(nq) < 0.12, 2, :] = _f32_cells([-0.0, 0.0])      # only the zeros
    r[rng.random(nq) < 0.12, 2, :] = _f32_cells([0.0, -0.0])
    r[rng.random(nq) < 0.12, 2, :] = _f32_cells([-np.inf, np.inf])
    return x, a, types, adj, entry, orc, q, r


@pytest.mark.parametrize("dtype,d,R", [("u8", 128, 32), ("f32", 32, 16)])
def test_attribute_edge_values(dtype, d, R):
    boa = _boa()
    x, a, types, adj, entry, orc, q, r = _edge_case_inputs(dtype, d, R, seed=d + R)
    valid = np.array([[oracle.phi(a[i], r[t], types) == 0 for i in range(0, a.shape[0], 7)]
                      for t in range(0, q.shape[0], 8)])
    assert 0.0 < valid.mean() < 1.0 and (~valid.any(1)).any()   # both kinds of valid set occur
    gpu = boa.Index(x, a, types, adj, entry)
    sched = oracle.schedule(16, 2.0, 128)
    ref = oracle.boa(orc, q, r, 10, sched, eps=0.1)
    for kw in ({}, {"fused": True}, {"split": True}):
        got = gpu_search(gpu, q, r, k=10, L0=16, Lmax=128, eps=0.1, **kw)
        assert_parity(got, ref, f"edge values {dtype} {kw}")
    ref_w = oracle.boa_warm(orc, q, r, 10, sched, eps=0.1)
    got = gpu_search(gpu, q, r, k=10, L0=16, Lmax=128, eps=0.1, fused=True, warm=True)
    assert_parity(got, ref_w, f"edge values {dtype} warm")
    ref = oracle.boa(orc, q, r, 10, [200])
    got = gpu_search(gpu, q, r, k=10, fixed_L=200)
    assert_parity(got, ref, f"edge values {dtype} fixed 200")
    gpu.close()


@pytest.mark.parametrize("eps", [0.0, 1.0])
def test_split_all_or_no_survivors(tiny, eps):
    """eps = 0 sends every query with more than k valid entries on to the
    wider phases (the escalation launch cannot hold them all at once and
    falls back to the default table); eps = 1 with unconstrained ranges
    leaves no survivor, so the escalation launch is skipped."""
    wl, d = tiny["wl"], tiny["data"]
    r = d.ranges.copy()
    if eps == 1.0:
        r[:, :, 0] = np.iinfo(np.int32).min
        r[:, :, 1] = np.iinfo(np.int32).max
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa(tiny["orc"], d.queries, r, wl.k, sched, eps=eps)
    got = gpu_search(tiny["gpu"], d.queries, r, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, eps=eps, split=True)
    assert_parity(got, ref, f"split eps={eps}")
    st = tiny["gpu"].stats()
    survivors = int((ref.final_L > wl.L0).sum())
    assert (survivors == 0) == (eps == 1.0)
    assert st["phases"][0]["launches"] == 1
    assert st["phases"][1]["launches"] == (1 if survivors else 0)


# ---------------------------------------------------------------------------
# the hand-traced golden graph (tests/golden/beam_trace.txt): the kernel's
# final results, widths and counts equal the values worked by hand

def test_hand_traced_golden():
    import os
    from helpers import load_beam_trace
    x, a, adj, entry, queries, searches, boas, warms = load_beam_trace(
        os.path.join(os.path.dirname(__file__), "golden", "beam_trace.txt"))
    gpu = _boa().Index(x, a, np.zeros(1, np.int32), adj, entry)
    for c in searches:
        # single width: the valid entries of the traced worklist, in order
        q, r = queries[c["q"]]
        valid = [(i, d) for i, p, d in zip(c["ids"], c["phi"], c["d"]) if p == 0]
        ids, dists, fl, E, S = gpu_search(gpu, q, r, k=len(valid), fixed_L=c["L"])
        assert ids[0].tolist() == [i for i, _ in valid], c
        assert dists[0].tolist() == [d for _, d in valid], c
        assert (fl[0], E[0], S[0]) == (c["L"], c["E"], c["S"]), c
    for c in boas:
        q, r = queries[c["q"]]
        for mode in MODES.values():
            ids, dists, fl, E, S = gpu_search(gpu, q, r, k=c["k"], schedule=c["widths"], eps=c["eps"], **mode)
            n = len(c["ids"])
            assert ids[0, :n].tolist() == c["ids"] and (ids[0, n:] == PAD).all(), (c, mode)
            assert dists[0, :n].tolist() == c["d"], (c, mode)
            assert (fl[0], E[0], S[0]) == (c["final_L"], c["E"], c["S"]), (c, mode)
    for c in warms:
        q, r = queries[c["q"]]
        ids, dists, fl, E, S = gpu_search(gpu, q, r, k=c["k"], schedule=c["widths"], eps=c["eps"],
                                          fused=True, warm=True)
        n = len(c["ids"])
        assert ids[0, :n].tolist() == c["ids"] and (ids[0, n:] == PAD).all(), c
        assert dists[0, :n].tolist() == c["d"], c
        assert (fl[0], E[0], S[0]) == (c["final_L"], c["E"], c["S"]), c
    gpu.close()


# ---------------------------------------------------------------------------
# warm-start escalation (fused mode) against the oracle's mirror mode

@pytest.mark.parametrize("eps", [0.0, 0.02, 0.05, 0.2])
def test_tiny_warm(tiny, eps):
    wl, d = tiny["wl"], tiny["data"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa_warm(tiny["orc"], d.queries, d.ranges, wl.k, sched, eps=eps)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, eps=eps,
                     fused=True, warm=True)
    assert_parity(got, ref, f"tiny warm eps={eps}")
    st = tiny["gpu"].stats()
    for p, rp in zip(st["phases"], ref.phases):
        assert (p["active"], p["confident"], p["expansions"], p["scored"]) == \
            (rp["active"], rp["confident"], rp["expansions"], rp["scored"])


@pytest.mark.parametrize("slots", [64, 256])
def test_warm_forced_spill(tiny, slots):
    """The visited set carried from phase to phase, with most inserts in the
    HBM bitmap (which must then not be reset by a continuing phase)."""
    wl, d = tiny["wl"], tiny["data"]
    sched = oracle.schedule(wl.L0, 2.0, wl.Lmax)
    ref = oracle.boa_warm(tiny["orc"], d.queries, d.ranges, wl.k, sched, eps=0.01)
    got = gpu_search(tiny["gpu"], d.queries, d.ranges, k=wl.k, L0=wl.L0, Lmax=wl.Lmax, eps=0.01,
                     fused=True, warm=True, lds_hash_slots=slots)
    assert_parity(got, ref, f"warm spill slots={slots}")
    assert tiny["gpu"].stats()["spilled_queries"] > 0


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{s[0]}-d{s[1]}-m{s[2]}-R{s[3]}" for s in SHAPES])
def test_shapes_warm(shape):
    dtype, d, m, R, f32col = shape
    boa = _boa()
    arrs = random_arrays(n=3000, d=d, m=m, R=R, dtype=dtype, seed=d + m + R, f32_col=f32col)
    orc = oracle.Index(*arrs)
    gpu = boa.Index(*arrs)
    q, r = random_queries(orc, 150, 40, seed=d, f32_col=f32col)
    for sched in (oracle.schedule(16, 2.0, 256), [10, 100, 200]):
        ref = oracle.boa_warm(orc, q, r, 10, sched, eps=0.05)
        got = gpu_search(gpu, q, r, k=10, schedule=sched, eps=0.05, fused=True, warm=True)
        assert_parity(got, ref, f"shape {shape} warm {sched}")
    gpu.close()


def test_warm_needs_the_fused_mode(tiny):
    boa = _boa()
    wl, d = tiny["wl"], tiny["data"]
    q = torch.from_numpy(d.queries[:4]).to("cuda:0")
    r = torch.from_numpy(d.ranges[:4]).to("cuda:0")
    for mode in ({}, {"split": True}, {"boa_plus": True}):
        with pytest.raises(boa.BoaError) as e:
            tiny["gpu"].search(q, r, k=wl.k, warm=True, **mode)
        assert e.value.code == -4
