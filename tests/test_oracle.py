"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every check here compares the oracle with something other than itself:
float64 arithmetic, exact integer arithmetic, hand-computed values from
the paper's definitions, exhaustive search, or structural invariants of
beam search (Sec. II "Beam search", Alg. 1, Alg. 2, Eqs. 1-3).
"""
import os

import numpy as np
import pytest

import oracle
from workloads import gen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


from helpers import (I32_MAX, I32_MIN, PAD, assert_same_up_to_near_ties, load_beam_trace,
                     numpy_filtered_topk, numpy_valid, random_index, random_queries, ring_knn_graph)


# ---------------------------------------------------------------------------
# distance

@pytest.mark.parametrize("d", [4, 8, 32, 96, 128, 200, 768])
def test_dist_f32_close_to_float64(d):
    rng = np.random.default_rng(d)
    for _ in range(50):
        x = rng.normal(size=d).astype(np.float32)
        q = rng.normal(size=d).astype(np.float32)
        ref = ((x.astype(np.float64) - q.astype(np.float64)) ** 2).sum()
        got = oracle.dist(x, q)
        assert abs(got - ref) <= 1e-6 * ref + 1e-30


def test_dist_f32_every_dimension_counts():
    # a dropped or misindexed term changes the sum: perturb each dim alone
    d = 96
    q = np.zeros(d, dtype=np.float32)
    for i in range(d):
        x = np.zeros(d, dtype=np.float32)
        x[i] = 3.0
        assert oracle.dist(x, q) == 9.0
        x[i] = -2.0
        assert oracle.dist(x, q) == 4.0


def test_dist_exact_on_integer_valued_data():
    rng = np.random.default_rng(7)
    for d in (32, 128):
        for _ in range(100):
            x = rng.integers(0, 256, size=d)
            q = rng.integers(0, 256, size=d)
            ref = int(((x - q) ** 2).sum())
            assert oracle.dist(x.astype(np.float32), q.astype(np.float32)) == ref
            assert oracle.dist(x.astype(np.uint8), q.astype(np.uint8)) == ref


def test_dist_u8_extremes():
    d = 128
    x = np.full(d, 255, dtype=np.uint8)
    q = np.zeros(d, dtype=np.uint8)
    assert oracle.dist(x, q) == d * 255 * 255
    assert oracle.dist(q, x) == d * 255 * 255
    assert oracle.dist(x, x) == 0


# ---------------------------------------------------------------------------
# filter distance phi (Eq. 2; JAG paragraph of Sec. II)

def test_phi_inclusive_bounds_and_counts():
    t = np.array([0, 0, 0], dtype=np.int32)
    r = np.array([[10, 20], [-5, -5], [0, 100]], dtype=np.int32)
    assert oracle.phi([10, -5, 0], r, t) == 0      # lower bounds are inclusive
    assert oracle.phi([20, -5, 100], r, t) == 0    # upper bounds are inclusive
    assert oracle.phi([9, -5, 50], r, t) == 1
    assert oracle.phi([21, -4, 50], r, t) == 2
    assert oracle.phi([9, -6, 101], r, t) == 3
    assert oracle.phi([I32_MIN, I32_MAX, 5], [[I32_MIN, I32_MAX]] * 3, t) == 0


def test_phi_float_column_compares_as_float():
    t = np.array([gen.ATTR_F32, gen.ATTR_I32], dtype=np.int32)
    r = np.zeros((2, 2), dtype=np.int32)
    r[0] = gen.f32_bits([-2.0, -1.0])
    r[1] = [0, 9]
    a = np.zeros(2, dtype=np.int32)
    for v, want in [(-1.5, 0), (-2.0, 0), (-1.0, 0), (-0.5, 1), (-2.5, 1), (0.0, 1)]:
        a[0] = gen.f32_bits([v])[0]
        a[1] = 3
        assert oracle.phi(a, r, t) == want, v
    # signed-integer comparison of the bit patterns would get these wrong
    a[0] = gen.f32_bits([-1.5])[0]
    assert oracle.phi(a, r, t) == 0
    inf = np.zeros((2, 2), dtype=np.int32)
    inf[0] = gen.f32_bits([-np.inf, np.inf])
    inf[1] = [I32_MIN, I32_MAX]
    a[0] = gen.f32_bits([1e30])[0]
    assert oracle.phi(a, inf, t) == 0


def test_phi_float_special_values_follow_ieee():
    """Zeros of both signs compare equal, NaN satisfies no bound (nor does any
    value a NaN bound), infinities and denormals order as numbers: every
    (value, lo, hi) triple over these cells against numpy's float32 compares."""
    cells = np.concatenate([
        gen.f32_bits([0.0, -0.0, np.inf, -np.inf, 1e-45, -1e-45, 3.4028235e38, -3.4028235e38, 1.0, -2.5]),
        np.array([0x7FC00000, 0xFFC00000, 0x7F800001], dtype=np.uint32).view(np.int32)])
    f = cells.view(np.float32)
    t = np.array([gen.ATTR_F32], dtype=np.int32)
    for i in range(cells.size):
        for j in range(cells.size):
            for k in range(cells.size):
                want = 0 if (f[j] <= f[i]) and (f[i] <= f[k]) else 1
                assert oracle.phi(cells[i:i + 1], [[cells[j], cells[k]]], t) == want, (f[i], f[j], f[k])
    z = gen.f32_bits([0.0, -0.0])
    assert oracle.phi(z[1:], [[z[0], z[0]]], t) == 0 and oracle.phi(z[:1], [[z[1], z[1]]], t) == 0


# ---------------------------------------------------------------------------
# confidence test (Eq. 3), golden cases

def _golden_confidence():
    cases = []
    with open(os.path.join(GOLDEN, "confidence_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            p = line.split()
            cases.append((int(p[0]), float(p[1]), bool(int(p[2])), [float(v) for v in p[3:]]))
    return cases


@pytest.mark.parametrize("case", _golden_confidence())
def test_confidence_golden(case):
    k, eps, want, D = case
    sq = np.array(D, dtype=np.float64) ** 2
    assert oracle.confident(sq.astype(np.float32), k, eps) == want


def test_confidence_monotone_in_eps():
    rng = np.random.default_rng(3)
    for _ in range(200):
        D = np.sort(rng.random(12) * 10).astype(np.float32)
        sq = (D.astype(np.float64) ** 2).astype(np.float32)
        g = (np.sqrt(np.float64(sq[-1])) - np.sqrt(np.float64(sq[4]))) / np.sqrt(np.float64(sq[-1]))
        assert oracle.confident(sq, 5, g * (1 + 1e-9)) is True
        assert oracle.confident(sq, 5, g * (1 - 1e-6)) is False


# ---------------------------------------------------------------------------
# beam schedule (Alg. 1: L grows by alpha; clamped at Lmax)

def test_schedule():
    assert oracle.schedule(16, 2.0, 512) == [16, 32, 64, 128, 256, 512]
    assert oracle.schedule(16, 2.0, 128) == [16, 32, 64, 128]
    assert oracle.schedule(16, 2.0, 1024) == [16, 32, 64, 128, 256, 512, 1024]
    assert oracle.schedule(10, 1.5, 40) == [10, 15, 23, 35, 40]
    assert oracle.schedule(16, 2.0, 100) == [16, 32, 64, 100]
    assert oracle.schedule(500, 2.0, 500) == [500]


# ---------------------------------------------------------------------------
# beam search at full width equals exhaustive filtered search (Def. 1)

@pytest.mark.parametrize("dtype,width,f32col", [("f32", 100, False), ("f32", 50, False),
                                                ("f32", 10, True), ("u8", 30, False),
                                                ("u8", 3, False)])
def test_full_width_search_is_exact(dtype, width, f32col):
    ix = random_index(n=300, d=16, m=2, R=10, dtype=dtype, seed=width, f32_col=f32col)
    q, r = random_queries(ix, 12, width, seed=width, f32_col=f32col)
    k = 10
    res = oracle.boa(ix, q, r, k, [ix.n])
    bi, bd, nv = oracle.bruteforce(ix, q, r, k)
    # same distance function: exact agreement with exhaustive search
    np.testing.assert_array_equal(res.ids, bi)
    np.testing.assert_array_equal(res.dists, bd)
    # every node reachable (the graph has a ring), nothing truncated:
    # every node is scored once and expanded once
    assert (res.expansions == ix.n).all() and (res.scored == ix.n).all()
    # and against an independent float64 evaluation of Def. 1
    for i in range(q.shape[0]):
        ri, rd = numpy_filtered_topk(ix, q[i], r[i], k)
        assert nv[i] == numpy_valid(ix, r[i]).sum()
        assert_same_up_to_near_ties(res.ids[i], res.dists[i].astype(np.float64), ri, rd)


def test_full_width_unfiltered_is_plain_knn():
    ix = random_index(n=250, d=32, m=1, R=8, seed=11)
    q, r = random_queries(ix, 10, 100, seed=11)
    r[:, :, 0], r[:, :, 1] = I32_MIN, I32_MAX      # g == 1 (Sec. II)
    res = oracle.boa(ix, q, r, 10, [ix.n])
    for i in range(q.shape[0]):
        d = ((ix.vectors.astype(np.float64) - q[i].astype(np.float64)) ** 2).sum(1)
        o = np.lexsort((np.arange(ix.n), d))[:10]
        assert_same_up_to_near_ties(res.ids[i], res.dists[i].astype(np.float64), o, d[o])


def test_fewer_valid_than_k_returns_all_valid():
    ix = random_index(n=200, d=8, m=1, R=8, seed=5)
    q, r = random_queries(ix, 6, 100, seed=5)
    a = ix.attrs[:, 0]
    vals = np.unique(a)
    for i in range(6):   # a range holding one attribute value: a handful of points
        r[i, 0] = [vals[i], vals[i]]
    res = oracle.boa(ix, q, r, 10, [ix.n])
    for i in range(6):
        ok = np.flatnonzero(a == vals[i])
        got = res.ids[i][res.ids[i] != PAD]
        assert sorted(got.tolist()) == sorted(ok.tolist()) or len(ok) > 10
        if len(ok) < 10:
            assert (res.ids[i][len(ok):] == PAD).all()
            assert np.isinf(res.dists[i][len(ok):]).all()


def test_empty_valid_set():
    ix = random_index(n=120, d=8, m=1, R=6, seed=9)
    q, r = random_queries(ix, 3, 100, seed=9)
    r[:, 0] = [1000, 2000]
    res = oracle.boa(ix, q, r, 10, [16, 32])
    assert (res.ids == PAD).all() and np.isinf(res.dists).all()
    assert (res.final_L == 32).all()          # never confident: runs to the last width


# ---------------------------------------------------------------------------
# narrow widths, pinned by hand-traced searches (Sec. II "Beam search",
# Alg. 2): which unexpanded entry goes next, merge-then-cut, exact seen-set
# semantics, distance ties by id, padded rows, valid points reached only
# through invalid ones, and the exact expansion and scored counts

_TRACE = load_beam_trace(os.path.join(GOLDEN, "beam_trace.txt"))


def _trace_index():
    x, a, adj, entry = _TRACE[:4]
    return oracle.Index(x, a, np.zeros(1, np.int32), adj, entry)


@pytest.mark.parametrize("case", _TRACE[5], ids=lambda c: f"{c['q']}-L{c['L']}")
def test_search_matches_hand_trace(case):
    ix = _trace_index()
    q, r = _TRACE[4][case["q"]]
    ids, ph, d, ln, E, S = oracle.search_lists(ix, q, r, case["L"])
    n = len(case["ids"])
    assert ln[0] == n
    assert ids[0, :n].tolist() == case["ids"]
    assert ph[0, :n].tolist() == case["phi"]
    assert d[0, :n].tolist() == case["d"]
    assert (E[0], S[0]) == (case["E"], case["S"])


@pytest.mark.parametrize("case", _TRACE[6], ids=lambda c: f"{c['q']}-k{c['k']}-eps{c['eps']}")
def test_boa_matches_hand_trace(case):
    ix = _trace_index()
    q, r = _TRACE[4][case["q"]]
    res = oracle.boa(ix, q, r, case["k"], case["widths"], eps=case["eps"])
    n = len(case["ids"])
    assert res.ids[0, :n].tolist() == case["ids"] and (res.ids[0, n:] == PAD).all()
    assert res.dists[0, :n].tolist() == case["d"]
    assert (res.final_L[0], res.expansions[0], res.scored[0]) == (case["final_L"], case["E"], case["S"])


# ---------------------------------------------------------------------------
# warm-start escalation (Sec. III-A "Redundancy Avoidance"; reading in the
# oracle's orc_boa_warm): hand-traced cases, and what the reading fixes

@pytest.mark.parametrize("case", _TRACE[7], ids=lambda c: f"{c['q']}-k{c['k']}-warm")
def test_warm_matches_hand_trace(case):
    ix = _trace_index()
    q, r = _TRACE[4][case["q"]]
    res = oracle.boa_warm(ix, q, r, case["k"], case["widths"], eps=case["eps"])
    n = len(case["ids"])
    assert res.ids[0, :n].tolist() == case["ids"] and (res.ids[0, n:] == PAD).all()
    assert res.dists[0, :n].tolist() == case["d"]
    assert (res.final_L[0], res.expansions[0], res.scored[0]) == (case["final_L"], case["E"], case["S"])


def test_warm_first_phase_is_the_restart_search(mid_index):
    """Phase 0 of the warm mode keeps a longer list but expands only among
    its first L0 entries: its worklist, and so every query that settles
    there, equal the fresh width-L0 search (results, E and S)."""
    ix = mid_index
    q, r = random_queries(ix, 60, 30, seed=41, f32_col=True)
    sched = oracle.schedule(10, 2.0, 160)
    # k = 5 < L0: a width-10 worklist can hold more valid entries than k,
    # so queries can settle at the first width (n_valid <= k never does)
    warm = oracle.boa_warm(ix, q, r, 5, sched, eps=0.3)
    cold = oracle.boa(ix, q, r, 5, sched, eps=0.3)
    assert warm.phases[0] == cold.phases[0]
    first = cold.final_L == sched[0]
    assert first.any() and (~first).any()
    np.testing.assert_array_equal(warm.final_L[first], cold.final_L[first])
    for a, b in ((warm.ids, cold.ids), (warm.dists, cold.dists), (warm.expansions, cold.expansions),
                 (warm.scored, cold.scored)):
        np.testing.assert_array_equal(a[first], b[first])
    # the escalated ones stop at the same widths (the test sees each phase's
    # worklist) only by coincidence; but they never score a node twice: at
    # most every point once over all phases
    assert (warm.scored <= ix.n).all()
    assert (warm.scored[~first] < cold.scored[~first]).mean() > 0.5


def test_warm_two_widths_ending_at_n_is_exact():
    """With widths [L0, N >= n] the first phase keeps up to N candidates,
    so nothing is ever cut and the last phase expands every reachable
    node: the result is the exact filtered top-k (Def. 1)."""
    ix = random_index(n=300, d=16, m=2, R=10, seed=43, f32_col=True)
    q, r = random_queries(ix, 15, 40, seed=43, f32_col=True)
    res = oracle.boa_warm(ix, q, r, 10, [10, ix.n], eps=0.0)
    bi, bd, nv = oracle.bruteforce(ix, q, r, 10)
    esc = res.final_L == ix.n
    assert esc.any()
    np.testing.assert_array_equal(res.ids[esc], bi[esc])
    np.testing.assert_array_equal(res.dists[esc], bd[esc])
    assert (res.scored[esc] == ix.n).all()   # every node scored exactly once


def test_warm_result_invariants(mid_index):
    ix = mid_index
    q, r = random_queries(ix, 50, 25, seed=44, f32_col=True)
    sched = oracle.schedule(16, 2.0, 256)
    res = oracle.boa_warm(ix, q, r, 10, sched, eps=0.05)
    for i in range(q.shape[0]):
        assert res.final_L[i] in sched
        got = res.ids[i][res.ids[i] != PAD]
        assert numpy_valid(ix, r[i])[got.astype(np.int64)].all()
        dd = res.dists[i][:len(got)]
        assert list(zip(dd, got)) == sorted(zip(dd, got))
        assert len(set(got.tolist())) == len(got)
        for j, g in enumerate(got):
            assert dd[j] == oracle.dist(ix.vectors[g], q[i])
    assert sum(p["expansions"] for p in res.phases) == res.expansions.sum()
    assert sum(p["scored"] for p in res.phases) == res.scored.sum()


# ---------------------------------------------------------------------------
# invariants at narrow widths (truncation active)

@pytest.fixture(scope="module")
def mid_index():
    return random_index(n=1500, d=32, m=2, R=12, seed=21, f32_col=True)


def test_worklist_invariants(mid_index):
    ix = mid_index
    q, r = random_queries(ix, 40, 40, seed=21, f32_col=True)
    for L in (10, 16, 37, 64):
        ids, ph, d, ln, E, S = oracle.search_lists(ix, q, r, L)
        for i in range(q.shape[0]):
            n = ln[i]
            assert 1 <= n <= L
            assert n == min(L, S[i])            # the beam is full whenever S >= L
            assert (ids[i, n:] == PAD).all()
            keys = list(zip(ph[i, :n], d[i, :n], ids[i, :n]))
            assert keys == sorted(keys)         # ascending (phi, d, id)
            assert len(set(ids[i, :n].tolist())) == n
            valid = numpy_valid(ix, r[i])
            np.testing.assert_array_equal(ph[i, :n] == 0, valid[ids[i, :n].astype(np.int64)])
            for j in range(n):                  # stored distance is the point's distance
                assert d[i, j] == oracle.dist(ix.vectors[ids[i, j]], q[i])
            assert 1 <= E[i] <= S[i] <= 1 + E[i] * ix.adj.shape[1]


def test_boa_result_invariants(mid_index):
    ix = mid_index
    q, r = random_queries(ix, 60, 30, seed=22, f32_col=True)
    sched = oracle.schedule(10, 2.0, 160)
    res = oracle.boa(ix, q, r, 10, sched, eps=0.2)
    assert len({int(v) for v in res.final_L}) >= 3      # several phases resolve queries
    for i in range(q.shape[0]):
        assert res.final_L[i] in sched
        got = res.ids[i][res.ids[i] != PAD]
        assert (res.ids[i][len(got):] == PAD).all()
        valid = numpy_valid(ix, r[i])
        assert valid[got.astype(np.int64)].all()          # every id satisfies all m predicates
        dd = res.dists[i][:len(got)]
        assert list(zip(dd, got)) == sorted(zip(dd, got))  # ascending by (d, id)
        assert len(set(got.tolist())) == len(got)
    # phases: active counts shrink by the confident counts
    ph = res.phases
    for a, b in zip(ph, ph[1:]):
        assert b["active"] == a["active"] - a["confident"]
    assert ph[0]["active"] == q.shape[0]
    assert sum(p["expansions"] for p in ph) == res.expansions.sum()


def test_restart_semantics(mid_index):
    """Each phase searches afresh, so query i's BOA result equals a
    single-width search at its final width (Alg. 1 calls Alg. 2 anew)."""
    ix = mid_index
    q, r = random_queries(ix, 50, 25, seed=23, f32_col=True)
    sched = oracle.schedule(10, 2.0, 160)
    res = oracle.boa(ix, q, r, 10, sched, eps=0.2)
    for L in sched:
        sel = np.flatnonzero(res.final_L == L)
        if sel.size == 0:
            continue
        one = oracle.boa(ix, q[sel], r[sel], 10, [L])
        np.testing.assert_array_equal(one.ids, res.ids[sel])
        np.testing.assert_array_equal(one.dists, res.dists[sel])


def test_batch_independence_and_threads(mid_index):
    ix = mid_index
    q, r = random_queries(ix, 64, 35, seed=24, f32_col=True)
    sched = oracle.schedule(10, 2.0, 80)
    full = oracle.boa(ix, q, r, 10, sched, threads=4)
    single = oracle.boa(ix, q, r, 10, sched, threads=1)
    np.testing.assert_array_equal(full.ids, single.ids)
    np.testing.assert_array_equal(full.expansions, single.expansions)
    perm = np.random.default_rng(0).permutation(64)[:20]
    sub = oracle.boa(ix, q[perm], r[perm], 10, sched)
    np.testing.assert_array_equal(sub.ids, full.ids[perm])
    np.testing.assert_array_equal(sub.final_L, full.final_L[perm])
    np.testing.assert_array_equal(sub.scored, full.scored[perm])


def test_tau_stops_early(mid_index):
    ix = mid_index
    q, r = random_queries(ix, 40, 30, seed=25, f32_col=True)
    sched = oracle.schedule(10, 2.0, 160)
    full = oracle.boa(ix, q, r, 10, sched, eps=0.3)
    ph = full.phases
    assert len(ph) >= 3 and ph[1]["confident"] > 0
    # a residual fraction between phase 2's and phase 1's active share
    # stops the loop after phase 1
    tau = (ph[2]["active"] + 0.5) / 40
    cut = oracle.boa(ix, q, r, 10, sched, eps=0.3, tau=tau)
    assert len(cut.phases) == 2
    assert set(cut.final_L.tolist()) <= {sched[0], sched[1]}
    np.testing.assert_array_equal(cut.ids[full.final_L <= sched[1]],
                                  full.ids[full.final_L <= sched[1]])


def test_u8_and_f32_integer_data_agree():
    """Integer-valued float32 data and the same data as uint8 give the same
    exact distances, hence identical searches."""
    rng = np.random.default_rng(31)
    xu = rng.integers(0, 256, size=(600, 16)).astype(np.uint8)
    ixu = random_index(n=600, d=16, m=2, R=10, dtype="u8", seed=31)
    ixu = oracle.Index(xu, ixu.attrs, ixu.attr_dtypes, ring_knn_graph(xu, 10, 31), ixu.entry)
    ixf = oracle.Index(xu.astype(np.float32), ixu.attrs, ixu.attr_dtypes, ixu.adj, ixu.entry)
    q, r = random_queries(ixu, 30, 40, seed=31)
    a = oracle.boa(ixu, q, r, 10, [16, 32, 64])
    b = oracle.boa(ixf, q.astype(np.float32), r, 10, [16, 32, 64])
    np.testing.assert_array_equal(a.ids, b.ids)
    np.testing.assert_array_equal(a.dists, b.dists)
    np.testing.assert_array_equal(a.final_L, b.final_L)


# ---------------------------------------------------------------------------
# the average-beamwidth reading, pinned by the paper's own table

def test_lavg_is_mean_final_width():
    rows, ranges = [], {}
    with open(os.path.join(GOLDEN, "tab_split.txt")) as f:
        for line in f:
            p = line.split()
            if not p or p[0].startswith("#"):
                continue
            if p[0] == "RANGE":
                ranges[int(p[1])] = (int(p[2]), int(p[3]))
            else:
                pct = [0.0 if v == "-" else float(v) for v in p[2:5]]
                rows.append((p[0], int(p[1]), pct))
    widths = [10, 100, 200]
    for m, (lo, hi) in ranges.items():
        finals = [sum(pc * w for pc, w in zip(pct, widths)) / 100 for _, mm, pct in rows if mm == m]
        # the prose rounds loosely (22.5 -> "22", 57.0 -> "58"): within about one unit
        assert abs(min(finals) - lo) <= 1.1 and abs(max(finals) - hi) <= 1.1
    # the cumulative reading (sum of every phase's width) contradicts "77"
    yt4 = [pct for name, mm, pct in rows if name == "YouTube" and mm == 4][0]
    cumulative = (yt4[0] * 10 + yt4[1] * 110 + yt4[2] * 310) / 100
    assert cumulative > 100
