"""Proximity-graph construction for the synthetic workloads.

The search method takes the graph as a given input (the paper builds it
offline with Vamana plus JAG threshold pruning, Sec. II "Graph
construction"). This module is that offline step for the synthetic data,
and it is deliberately not the paper's builder:

  1. exact kNN candidates (2R per point, ordered by distance then id);
  2. relative-neighbourhood pruning with slack alpha (a candidate v is
     dropped when an already kept w satisfies alpha * d(w, v) <= d(u, v)),
     the DiskANN/Vamana diversification rule;
  3. a flat navigation layer: a seeded sample of points plus one
     representative per connected component of the pruned kNN graph.
     Each sample point links to sample points of other components, chosen
     by the same alpha-pruning (so roughly one per nearby component), and
     every point links to its nearest sample points. Clustered mixtures
     otherwise give one disconnected kNN component per cluster;
  4. random-subset levels: for a few fractions f, a seeded subset holding
     about f of the points, and every point's alpha-pruned nearest members
     of it. Their spacing grows as f shrinks, so these edges span the data
     at several scales whatever the attributes are;
  5. connectivity repair: every point is made reachable from the entry
     point (the point nearest the data centroid).

With attributes given, rows also carry attribute-aware edges in the manner
of JAG's threshold pruning (Sec. II "Graph construction"): each attribute
value is mapped to its quantile in its column, the attribute distance of
two points is the largest quantile gap over the columns, and for each of a
few thresholds t (per-point quantiles of the attribute distance to a
seeded sample) a point links, under its own degree budget, to the
alpha-pruned nearest vectors among the points within attribute distance t.
Under a narrow range predicate the valid points then keep edges among
themselves, which a valid-first search needs.

Rows are fixed-width n x R uint32 with 0xFFFFFFFF padding. Everything is
deterministic for a given device. Distances here are this module's own
(float64 on the CPU, float32 GEMM on a GPU) and share no code with either
search implementation.
"""
from __future__ import annotations

import math
import sys
import time

import numpy as np
import torch

PAD = 0xFFFFFFFF


def _log(msg: str):
    print(f"[graph {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def _as_float(x: np.ndarray, dev: torch.device) -> torch.Tensor:
    dt = torch.float64 if dev.type == "cpu" else torch.float32
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev).to(dt)


def entry_point(vectors: np.ndarray) -> int:
    """Id of the point nearest (float64 L2) to the float64 centroid; lowest id on ties."""
    n = vectors.shape[0]
    c = np.zeros(vectors.shape[1], dtype=np.float64)
    step = 1 << 16
    for s in range(0, n, step):
        c += vectors[s:s + step].astype(np.float64).sum(axis=0)
    c /= n
    best, best_d = -1, np.inf
    for s in range(0, n, step):
        x = vectors[s:s + step].astype(np.float64)
        dd = ((x - c) ** 2).sum(axis=1)
        j = int(np.argmin(dd))
        if dd[j] < best_d:
            best, best_d = s + j, float(dd[j])
    return best


def _sq_dist(a: torch.Tensor, b: torch.Tensor, na: torch.Tensor, nb: torch.Tensor) -> torch.Tensor:
    d = na[:, None] + nb[None, :] - 2.0 * (a @ b.T)
    return d.clamp_min_(0)


def _sort_by_dist_then_id(dist: torch.Tensor, ids: torch.Tensor):
    o = torch.argsort(ids, dim=1, stable=True)
    dist, ids = dist.gather(1, o), ids.gather(1, o)
    o = torch.argsort(dist, dim=1, stable=True)
    return dist.gather(1, o), ids.gather(1, o)


def knn(X: torch.Tensor, K: int, targets: torch.Tensor | None = None, exclude_self=True,
        chunk: int = 4096, mask_fn=None):
    """K nearest rows of `targets` (default X) for every row of X; (dist, ids) sorted.
    mask_fn(s, e) -> bool (e-s) x T marks targets to exclude for rows s..e."""
    T = X if targets is None else targets
    nx = (X * X).sum(1)
    nt = nx if targets is None else (T * T).sum(1)
    n = X.shape[0]
    out_d = torch.empty((n, K), dtype=X.dtype, device=X.device)
    out_i = torch.empty((n, K), dtype=torch.int64, device=X.device)
    extra = 4  # margin so ties at the boundary resolve by id
    kk = min(K + extra + (1 if exclude_self else 0), T.shape[0])
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        D = _sq_dist(X[s:e], T, nx[s:e], nt)
        if exclude_self:
            r = torch.arange(s, e, device=X.device)
            D[r - s, r] = float("inf")
        if mask_fn is not None:
            D.masked_fill_(mask_fn(s, e), float("inf"))
        dv, di = torch.topk(D, kk, dim=1, largest=False, sorted=True)
        dv, di = _sort_by_dist_then_id(dv, di)
        out_d[s:e], out_i[s:e] = dv[:, :K], di[:, :K]
        del D
    return out_d, out_i


def alpha_prune(X: torch.Tensor, cand: torch.Tensor, du: torch.Tensor, valid: torch.Tensor,
                budget: torch.Tensor, alpha: float, chunk: int = 0) -> torch.Tensor:
    """Greedy diversification of each row's sorted candidates; returns keep mask.
    Rows are independent; `chunk` only bounds the temporaries."""
    n, K = cand.shape
    if chunk <= 0:
        chunk = 8192 if n <= 2_000_000 or X.device.type == "cpu" else 65536
    keep_all = torch.zeros((n, K), dtype=torch.bool, device=X.device)
    a2 = alpha * alpha
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        c = cand[s:e].clamp_min(0)
        V = X[c]                                   # B x K x d
        nv = (V * V).sum(-1)
        G = torch.bmm(V, V.transpose(1, 2).contiguous())
        Dvv = (nv[:, :, None] + nv[:, None, :] - 2.0 * G).clamp_min_(0)
        dus = du[s:e]
        val = valid[s:e]
        bud = budget[s:e]
        keep = torch.zeros((e - s, K), dtype=torch.bool, device=X.device)
        cnt = torch.zeros(e - s, dtype=torch.int64, device=X.device)
        for j in range(K):
            if j > 0:
                dom = (keep[:, :j] & (a2 * Dvv[:, :j, j] <= dus[:, j:j + 1])).any(1)
            else:
                dom = torch.zeros(e - s, dtype=torch.bool, device=X.device)
            ok = val[:, j] & ~dom & (cnt < bud)
            keep[:, j] = ok
            cnt += ok.to(torch.int64)
        keep_all[s:e] = keep
        del V, G, Dvv
    return keep_all


def _with_reverse(cand, du, keep, width):
    """Each row's kept candidates plus the rows that kept it (closest first),
    deduplicated, sorted by (distance, id), cut to `width` (missing = inf)."""
    n, K = cand.shape
    dev = cand.device
    src = torch.arange(n, device=dev)[:, None].expand(n, K)[keep]
    dst = cand[keep]
    dd = du[keep]
    # group reverse edges by destination, nearest first, at most `width` each
    o = torch.argsort(dd, stable=True)
    src, dst, dd = src[o], dst[o], dd[o]
    o = torch.argsort(dst, stable=True)
    src, dst, dd = src[o], dst[o], dd[o]
    start = torch.zeros(n + 1, dtype=torch.int64, device=dev)
    start[1:] = torch.cumsum(torch.bincount(dst, minlength=n), 0)
    rank = torch.arange(dst.numel(), device=dev) - start[dst]
    ok = rank < width
    rev_i = torch.full((n, width), -1, dtype=torch.int64, device=dev)
    rev_d = torch.full((n, width), float("inf"), dtype=du.dtype, device=dev)
    rev_i[dst[ok], rank[ok]] = src[ok]
    rev_d[dst[ok], rank[ok]] = dd[ok]
    fw_i = torch.where(keep, cand, torch.full_like(cand, -1))
    fw_d = torch.where(keep, du, torch.full_like(du, float("inf")))
    ids = torch.cat([fw_i, rev_i], 1)
    ds = torch.cat([fw_d, rev_d], 1)
    # dedupe: sort by id, drop repeats
    o = torch.argsort(ids, dim=1, stable=True)
    ids, ds = ids.gather(1, o), ds.gather(1, o)
    rep = torch.zeros_like(ids, dtype=torch.bool)
    rep[:, 1:] = ids[:, 1:] == ids[:, :-1]
    ds = torch.where(rep | (ids < 0), torch.full_like(ds, float("inf")), ds)
    ds, ids = _sort_by_dist_then_id(ds, ids.clamp_min(0))
    ids = torch.where(torch.isfinite(ds), ids, torch.full_like(ids, -1))
    return ids[:, :width], ds[:, :width]


def _compact(a: torch.Tensor, width: int) -> torch.Tensor:
    """Move the non-negative entries of each row to the front (order kept)."""
    o = torch.argsort((a < 0).to(torch.int8), dim=1, stable=True)
    return a.gather(1, o)[:, :width]


def _components(n: int, rows: np.ndarray) -> np.ndarray:
    from scipy.sparse import coo_matrix
    from scipy.sparse.csgraph import connected_components
    src = np.repeat(np.arange(n, dtype=np.int32), rows.shape[1])
    dst = rows.reshape(-1).astype(np.int32)
    ok = dst >= 0
    g = coo_matrix((np.ones(int(ok.sum()), dtype=np.int8), (src[ok], dst[ok])), shape=(n, n)).tocsr()
    _, lab = connected_components(g, directed=False)
    return lab


def _reachable(n: int, adj: np.ndarray, s: int) -> np.ndarray:
    from scipy.sparse import csr_matrix
    from scipy.sparse.csgraph import breadth_first_order
    R = adj.shape[1]
    a = adj.astype(np.int64)
    a[adj == PAD] = -1
    ok = a >= 0
    indptr = np.zeros(n + 1, dtype=np.int64)
    indptr[1:] = np.cumsum(ok.sum(1))
    g = csr_matrix((np.ones(int(ok.sum()), dtype=np.int8), a[ok], indptr), shape=(n, n))
    order = breadth_first_order(g, s, directed=True, return_predecessors=False)
    seen = np.zeros(n, dtype=bool)
    seen[order] = True
    return seen


def attribute_quantiles(attrs: np.ndarray, attr_dtypes) -> np.ndarray:
    """n x m float64: each cell's mid-rank in its column divided by n (ties
    share one value); float32 columns are ranked by value, not by bits."""
    from scipy.stats import rankdata
    n, m = attrs.shape
    out = np.empty((n, m), dtype=np.float64)
    for j in range(m):
        col = attrs[:, j]
        if int(attr_dtypes[j]) == 1:
            col = np.ascontiguousarray(col).view(np.float32)
        out[:, j] = (rankdata(col, method="average") - 0.5) / n
    return out


def _attr_dist(A: torch.Tensor, B: torch.Tensor) -> torch.Tensor:
    """Largest per-column quantile gap between rows of A and rows of B."""
    d = None
    for j in range(A.shape[1]):
        g = (A[:, j:j + 1] - B[None, :, j]).abs()
        d = g if d is None else torch.maximum(d, g)
    return d


def _thresholds(QA: torch.Tensor, levels, seed: int, chunk: int) -> torch.Tensor:
    """n x len(levels): per point, the given quantiles of its attribute
    distance to a seeded sample of points."""
    n = QA.shape[0]
    dev = QA.device
    g = np.random.Generator(np.random.PCG64(seed ^ 0x5A5A))
    S = min(n - 1, 4096)
    samp = torch.from_numpy(np.sort(g.choice(n, size=S, replace=False))).to(dev)
    thr = torch.empty((n, len(levels)), dtype=QA.dtype, device=dev)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        ds, _ = torch.sort(_attr_dist(QA[s:e], QA[samp]), dim=1)
        for li, lv in enumerate(levels):
            thr[s:e, li] = ds[:, min(S - 1, int(lv * S))]
    return thr


def candidates(X: torch.Tensor, K: int, QA: torch.Tensor | None = None, thr: torch.Tensor | None = None,
               K_attr: int = 0, chunk: int = 2048, member: torch.Tensor | None = None):
    """One exhaustive pass: every point's K nearest others (dist, ids) and its
    K_attr nearest within each level (levels x n x K_attr, missing = inf /
    unspecified id). The levels are, first, the attribute threshold levels
    (attribute quantiles QA, thresholds thr: n x levels; a target is in a
    level when its attribute distance is within the threshold), then the
    random-subset levels (member: levels x n bool). Sorted by (distance, id)."""
    n = X.shape[0]
    dev = X.device
    nx = (X * X).sum(1)
    kk = min(n, K + 5)
    du = torch.empty((n, K), dtype=X.dtype, device=dev)
    cand = torch.empty((n, K), dtype=torch.int64, device=dev)
    nl_a = 0 if thr is None else thr.shape[1]
    nl = nl_a + (0 if member is None else member.shape[0])
    ka = min(n, K_attr + 5)
    du_l = torch.empty((nl, n, K_attr), dtype=X.dtype, device=dev)
    cand_l = torch.empty((nl, n, K_attr), dtype=torch.int64, device=dev)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        D = _sq_dist(X[s:e], X, nx[s:e], nx)
        r = torch.arange(s, e, device=dev)
        D[r - s, r] = float("inf")
        dv, di = torch.topk(D, kk, dim=1, largest=False, sorted=True)
        dv, di = _sort_by_dist_then_id(dv, di)
        du[s:e], cand[s:e] = dv[:, :K], di[:, :K]
        if nl:
            A = _attr_dist(QA[s:e], QA) if nl_a else None
            for li in range(nl):
                out = A > thr[s:e, li:li + 1] if li < nl_a else ~member[li - nl_a][None, :]
                Dl = torch.where(out, torch.full_like(D, float("inf")), D)
                dv, di = torch.topk(Dl, ka, dim=1, largest=False, sorted=True)
                dv, di = _sort_by_dist_then_id(dv, di)
                du_l[li, s:e], cand_l[li, s:e] = dv[:, :K_attr], di[:, :K_attr]
                del Dl
            del A
        del D
    return du, cand, du_l, cand_l


def _nearest_centroids(X: torch.Tensor, cent: torch.Tensor, k: int, chunk: int = 65536) -> torch.Tensor:
    """n x k ids of each row's nearest centroids (squared L2, ties by id)."""
    nc = (cent * cent).sum(1)
    out = torch.empty((X.shape[0], k), dtype=torch.int64, device=X.device)
    for s in range(0, X.shape[0], chunk):
        e = min(X.shape[0], s + chunk)
        D = nc[None, :] - 2.0 * (X[s:e] @ cent.T)
        dv, di = torch.topk(D, min(cent.shape[0], k + 4), dim=1, largest=False, sorted=True)
        dv, di = _sort_by_dist_then_id(dv, di)
        out[s:e] = di[:, :k]
    return out


def kmeans(X: torch.Tensor, C: int, iters: int = 6, sample: int = 1 << 20, seed: int = 0):
    """Lloyd's k-means on a seeded sample (centroids start at sample points)."""
    n = X.shape[0]
    g = np.random.Generator(np.random.PCG64(seed ^ 0x1F1F))
    S = min(n, sample)
    idx = torch.from_numpy(np.sort(g.choice(n, size=S, replace=False))).to(X.device)
    Xs = X[idx]
    cent = Xs[torch.from_numpy(np.sort(g.choice(S, size=C, replace=False))).to(X.device)].clone()
    for _ in range(iters):
        a = _nearest_centroids(Xs, cent, 1)[:, 0]
        sums = torch.zeros_like(cent).index_add_(0, a, Xs)
        cnt = torch.bincount(a, minlength=C)
        nz = cnt > 0
        cent[nz] = sums[nz] / cnt[nz, None].to(X.dtype)
    return cent


def candidates_ivf(X: torch.Tensor, K: int, QA: torch.Tensor | None = None, thr: torch.Tensor | None = None,
                   K_attr: int = 0, lists: int = 0, nprobe: int = 16, seed: int = 0, batch_elems: int = 1 << 28,
                   member: torch.Tensor | None = None):
    """The outputs of `candidates`, searched per k-means list instead of
    exhaustively: the members of each list against the points of its
    `nprobe` nearest lists (itself included). Exact within that pool."""
    n, dev = X.shape[0], X.device
    C = lists if lists > 0 else max(1, min(16384, n // 1024))
    t0 = time.time()
    cent = kmeans(X, C, seed=seed)
    a = _nearest_centroids(X, cent, 1)[:, 0]
    order = torch.argsort(a, stable=True)
    cnt = torch.bincount(a, minlength=C)
    off = torch.zeros(C + 1, dtype=torch.int64, device=dev)
    off[1:] = torch.cumsum(cnt, 0)
    probe = _nearest_centroids(cent, cent, min(C, nprobe))        # C x nprobe (itself first)
    _log(f"ivf: {C} lists (sizes {int(cnt.min())}..{int(cnt.max())}), {probe.shape[1]} probed, "
         f"{time.time() - t0:.1f}s")
    nx = (X * X).sum(1)
    du = torch.full((n, K), float("inf"), dtype=X.dtype, device=dev)
    cand = torch.full((n, K), -1, dtype=torch.int64, device=dev)
    nl_a = 0 if thr is None else thr.shape[1]
    nl = nl_a + (0 if member is None else member.shape[0])
    du_l = torch.full((nl, n, K_attr), float("inf"), dtype=X.dtype, device=dev)
    cand_l = torch.full((nl, n, K_attr), -1, dtype=torch.int64, device=dev)
    cnt_h = cnt.cpu().numpy()
    off_h = off.cpu().numpy()
    probe_h = probe.cpu().numpy()
    psize = cnt_h[probe_h].sum(1)
    # lists in order of pool size, so that a batch pads little
    seq = np.lexsort((np.arange(C), cnt_h, psize))
    c0 = 0
    while c0 < C:
        # lists seq[c0:c1] padded to the batch's largest list and pool
        c1, mm, pm = c0, 0, 0
        while c1 < C:
            mm2, pm2 = max(mm, int(cnt_h[seq[c1]])), max(pm, int(psize[seq[c1]]))
            if c1 > c0 and (c1 - c0 + 1) * mm2 * pm2 > batch_elems:
                break
            mm, pm, c1 = mm2, pm2, c1 + 1
        B = c1 - c0
        mem = torch.full((B, mm), -1, dtype=torch.int64)
        pool = torch.full((B, pm), -1, dtype=torch.int64)
        for b, c in enumerate(seq[c0:c1]):
            mem[b, :cnt_h[c]] = torch.arange(off_h[c], off_h[c + 1])
            parts = [torch.arange(off_h[q], off_h[q + 1]) for q in probe_h[c]]
            pp = torch.cat(parts)
            pool[b, :pp.numel()] = pp
        mem, pool = mem.to(dev), pool.to(dev)
        mid = torch.where(mem >= 0, order[mem.clamp_min(0)], torch.full_like(mem, -1))
        pid = torch.where(pool >= 0, order[pool.clamp_min(0)], torch.full_like(pool, -1))
        Xm, Xp = X[mid.clamp_min(0)], X[pid.clamp_min(0)]
        D = nx[mid.clamp_min(0)][:, :, None] + nx[pid.clamp_min(0)][:, None, :] - 2.0 * torch.bmm(
            Xm, Xp.transpose(1, 2).contiguous())
        D.clamp_min_(0)
        bad = (pid < 0)[:, None, :] | (pid[:, None, :] == mid[:, :, None])
        D.masked_fill_(bad, float("inf"))
        ok_rows = mid >= 0
        rows = mid[ok_rows]

        def take(Dm, k_out, dst_d, dst_i):
            kk = min(Dm.shape[2], k_out + 5)
            dv, di = torch.topk(Dm, kk, dim=2, largest=False, sorted=True)
            ids = torch.gather(pid[:, None, :].expand(-1, Dm.shape[1], -1), 2, di)
            dv, ids = dv[ok_rows], ids[ok_rows]
            ids = torch.where(torch.isfinite(dv), ids, torch.full_like(ids, n))
            dv, ids = _sort_by_dist_then_id(dv, ids)
            ids = torch.where(torch.isfinite(dv), ids, torch.full_like(ids, -1))
            w = min(k_out, dv.shape[1])
            dst_d[rows, :w], dst_i[rows, :w] = dv[:, :w], ids[:, :w]

        take(D, K, du, cand)
        if nl:
            A = None
            if nl_a:
                for j in range(QA.shape[1]):
                    gj = (QA[mid.clamp_min(0), j][:, :, None] - QA[pid.clamp_min(0), j][:, None, :]).abs()
                    A = gj if A is None else torch.maximum(A, gj)
                th = thr[mid.clamp_min(0)]                      # B x mm x levels
            for li in range(nl):
                if li < nl_a:
                    out = A > th[:, :, li:li + 1]
                else:
                    out = ~member[li - nl_a][pid.clamp_min(0)][:, None, :]
                Dl = torch.where(out, torch.full_like(D, float("inf")), D)
                take(Dl, K_attr, du_l[li], cand_l[li])
                del Dl
            del A
        del D, Xm, Xp
        c0 = c1
    return du, cand, du_l, cand_l


def level_edges(X: torch.Tensor, du_l: torch.Tensor, cand_l: torch.Tensor, budgets, alpha: float) -> torch.Tensor:
    """n x sum(budgets) ids (-1 = none): per level, the alpha-pruned nearest
    vectors among the level's candidates, at most budgets[level] of them."""
    n = X.shape[0]
    out = []
    for li in range(du_l.shape[0]):
        b = int(budgets[li])
        keep = alpha_prune(X, cand_l[li], du_l[li], torch.isfinite(du_l[li]),
                           torch.full((n,), b, dtype=torch.int64, device=X.device), alpha)
        out.append(_compact(torch.where(keep, cand_l[li], torch.full_like(cand_l[li], -1)), b))
    return torch.cat(out, 1)


def build_graph(vectors: np.ndarray, R: int, device: str | torch.device = "cpu",
                alpha: float = 1.2, seed: int = 0x9A9A, entry: int | None = None,
                attrs: np.ndarray | None = None, attr_dtypes=None,
                attr_levels=(0.001, 0.01, 0.05, 0.2), attr_budget: int | None = None,
                sub_levels=(0.001, 0.01, 0.05), sub_budget: int | None = None,
                cross_links: int | None = None, exact_limit: int = 2_000_000):
    """Fixed-degree proximity graph; returns (adjacency n x R uint32, entry id).
    Rows hold, besides the pruned nearest neighbours and the navigation
    links, `sub_budget` (default R // 32) edges per random-subset level (the
    alpha-pruned nearest members of a seeded subset holding that fraction of
    the points: edges at the scale of the subset's spacing) and, with
    `attrs` (n x m cells, column types `attr_dtypes`), `attr_budget`
    (default R // 6) attribute-aware edges per threshold level. The pruned
    nearest neighbours fill what the other links leave of a row. Above
    `exact_limit` points the candidates come from k-means lists
    (`candidates_ivf`) instead of an exhaustive pass."""
    dev = torch.device(device)
    n = vectors.shape[0]
    s_id = entry_point(vectors) if entry is None else int(entry)
    X = _as_float(vectors, dev)
    Kc = min(2 * R, n - 1)
    # 1-2: exact kNN candidates and, from the same distance pass, the
    # candidates of every random-subset level and attribute threshold level
    t0 = time.time()
    QA = thr = member = None
    budgets = []
    if attrs is not None and len(attr_levels) > 0:
        QA = _as_float(attribute_quantiles(attrs, attr_dtypes), dev)
        thr = _thresholds(QA, attr_levels, seed, 2048 if n <= exact_limit or dev.type == "cpu" else 32768)
        budgets += [max(1, R // 6) if attr_budget is None else int(attr_budget)] * len(attr_levels)
    n_attr_levels = len(budgets)
    if len(sub_levels) > 0:
        g = np.random.Generator(np.random.PCG64(seed ^ 0x3C3C))
        u = g.random((len(sub_levels), n))
        member = torch.from_numpy(u < np.asarray(sub_levels, dtype=np.float64)[:, None]).to(dev)
        budgets += [max(1, R // 32) if sub_budget is None else int(sub_budget)] * len(sub_levels)
    K_l = min(n - 1, 2 * max(budgets)) if budgets else 0
    if n > exact_limit:
        du, cand, du_l, cand_l = candidates_ivf(X, Kc, QA, thr, K_l, seed=seed, member=member)
    else:
        du, cand, du_l, cand_l = candidates(X, Kc, QA, thr, K_l, member=member)
    attr_e = None
    if budgets:
        # subset edges first in the row, then the attribute-aware ones
        lev = level_edges(X, du_l, cand_l, budgets, alpha)
        na = sum(budgets[:n_attr_levels])
        attr_e = torch.cat([lev[:, na:], lev[:, :na]], 1)
    del du_l, cand_l, QA, thr, member
    _log(f"{Kc}-NN candidates and level edges (budgets {budgets}) of {n} points in {time.time() - t0:.1f}s")
    R_cross = max(2, R // 8) if cross_links is None else int(cross_links)
    R_long = R_cross + 1
    K_nav = max(2, R // 2)

    # reverse edges (NSG/Vamana style): every kept edge u->v offers u to v.
    reserve = 1 if R >= 8 else 0   # one free slot per row for the connectivity repair
    n_attr = 0 if attr_e is None else attr_e.shape[1]
    base_budget = torch.full((n,), max(1, R - R_long - reserve - n_attr), dtype=torch.int64, device=dev)
    keep0 = alpha_prune(X, cand, du, torch.ones_like(cand, dtype=torch.bool), base_budget, alpha)
    cand, du = _with_reverse(cand, du, keep0, Kc)
    rows0 = torch.where(torch.isfinite(du), cand, torch.full_like(cand, -1)).cpu().numpy()
    _log(f"forward-pruned + reverse candidates ({time.time() - t0:.1f}s)")

    # 3: navigation sample (seeded sample + component representatives + entry).
    lab = _components(n, rows0)
    _log(f"pruned; {lab.max() + 1} components of the kNN graph ({time.time() - t0:.1f}s)")
    first_of = np.full(lab.max() + 1, n, dtype=np.int64)
    np.minimum.at(first_of, lab, np.arange(n))
    g = np.random.Generator(np.random.PCG64(seed))
    m0 = min(n, int(math.ceil(2 * math.sqrt(n))))
    P = np.unique(np.concatenate([first_of, g.choice(n, size=m0, replace=False), [s_id]]))
    Pt = torch.from_numpy(P).to(dev)
    XP = X[Pt]
    is_nav = torch.zeros(n, dtype=torch.bool, device=dev)
    is_nav[Pt] = True

    # sample-to-sample links: alpha-pruning over each sample's nearest
    # samples in OTHER components (the kNN graph already connects a
    # component internally), so each sample links to nearby components.
    KP = min(len(P) - 1, 256)
    dPP, iPP = knn(XP, KP)
    labP = torch.from_numpy(lab[P]).to(dev)
    lab_t = torch.from_numpy(lab).to(dev)
    other = labP[iPP] != labP[:, None]
    nav_keep = alpha_prune(XP, iPP, dPP, other,
                           torch.full((len(P),), K_nav, dtype=torch.int64, device=dev), alpha)
    nav_ids = _compact(torch.where(nav_keep, Pt[iPP], torch.full_like(iPP, -1)), K_nav)
    nav_links = torch.full((n, K_nav), -1, dtype=torch.int64, device=dev)
    nav_links[Pt] = nav_ids

    # every point: links to nearby components (alpha-pruned over its nearest
    # sample points of other components) and to its own component's nearest
    # sample point, so that every expansion also looks across components.
    Kx = min(len(P), 4 * R_cross)
    d_near, i_near = knn(X, Kx, targets=XP, exclude_self=False,
                         mask_fn=lambda s, e: labP[None, :] == lab_t[s:e, None])
    cross_keep = alpha_prune(XP, i_near, d_near, torch.isfinite(d_near),
                             torch.full((n,), R_cross, dtype=torch.int64, device=dev), alpha)
    cross = _compact(torch.where(cross_keep, Pt[i_near], torch.full_like(i_near, -1)), R_cross)
    d_own, i_own = knn(X, min(2, len(P)), targets=XP, exclude_self=False,
                       mask_fn=lambda s, e: labP[None, :] != lab_t[s:e, None])
    own = Pt[i_own]
    bad = (own == torch.arange(n, device=dev)[:, None]) | ~torch.isfinite(d_own)
    own = _compact(torch.where(bad, torch.full_like(own, -1), own), 1)
    near = torch.cat([cross, own], 1)
    _log(f"navigation: {len(P)} sample points, {R_cross} cross-component links per point")

    long = torch.cat([nav_links, near] + ([] if attr_e is None else [attr_e]), 1)
    dup = torch.zeros_like(long, dtype=torch.bool)
    for j in range(1, long.shape[1]):
        dup[:, j] = (long[:, :j] == long[:, j:j + 1]).any(1)
    self_l = long == torch.arange(n, device=dev)[:, None]
    long = _compact(torch.where(dup | self_l, torch.full_like(long, -1), long), long.shape[1])
    if long.shape[1] > R - reserve:
        long[:, R - reserve:] = -1
    n_long = (long >= 0).sum(1)

    # base candidates not already linked, pruned into the remaining budget.
    in_long = torch.zeros_like(cand, dtype=torch.bool)
    for j in range(long.shape[1]):
        in_long |= cand == long[:, j:j + 1]
    keep = alpha_prune(X, cand, du, ~in_long & torch.isfinite(du), R - n_long - reserve, alpha)

    adj = np.full((n, R), PAD, dtype=np.uint32)
    longn = long.cpu().numpy()
    candn = cand.cpu().numpy()
    keepn = keep.cpu().numpy()
    for_rows = np.full((n, R), -1, dtype=np.int64)
    # compact: long links first, then kept base candidates in distance order
    merged = np.concatenate([longn, np.where(keepn, candn, -1)], axis=1)
    order = np.argsort(merged < 0, axis=1, kind="stable")
    merged = np.take_along_axis(merged, order, axis=1)[:, :R]
    for_rows[:, :merged.shape[1]] = merged
    adj[for_rows >= 0] = for_rows[for_rows >= 0].astype(np.uint32)

    # 4: connectivity repair from the entry point.
    left = link_unreachable(adj, s_id, candn)
    _log(f"assembled rows; unreachable points linked in one pass, {left.size} left for the repair")
    if left.size:
        adj = repair(adj, vectors, s_id, P, candn)
    return adj, s_id


def link_unreachable(adj: np.ndarray, s_id: int, cand: np.ndarray) -> np.ndarray:
    """Give every point unreachable from s_id an in-edge from a reachable one,
    all at once: each such point proposes its candidates in distance order
    (a point's candidates are sorted nearest first); a reachable proposer
    target with a free (padding) slot accepts the lowest-id proposal of a
    round. Points left without a link are returned for the slower repair."""
    n, R = adj.shape
    seen = _reachable(n, adj, s_id)
    U = np.flatnonzero(~seen)
    if U.size == 0:
        return U
    free = (adj == PAD)
    nfree = free.sum(1)
    first_free = np.where(nfree > 0, np.argmax(free, axis=1), -1)
    C = cand[U]
    pending = np.ones(U.size, dtype=bool)
    for j in range(C.shape[1]):
        if not pending.any():
            break
        w = C[:, j]
        ok = pending & (w >= 0)
        ok[ok] = seen[w[ok]] & (nfree[w[ok]] > 0)
        if not ok.any():
            continue
        ui, wi = U[ok], w[ok]
        o = np.lexsort((ui, wi))               # per target, lowest proposer first
        ui, wi = ui[o], wi[o]
        lead = np.ones(wi.size, dtype=bool)
        lead[1:] = wi[1:] != wi[:-1]
        ui, wi = ui[lead], wi[lead]
        adj[wi, first_free[wi]] = ui.astype(np.uint32)
        nfree[wi] -= 1
        row = adj[wi] == PAD
        first_free[wi] = np.where(row.any(1), np.argmax(row, axis=1), -1)
        pending[np.searchsorted(U, ui)] = False
    return U[pending]


def repair(adj: np.ndarray, vectors: np.ndarray, s_id: int, P: np.ndarray,
           cand: np.ndarray, rounds: int = 32):
    """Make every point reachable from s_id.

    An unreachable point v gets an in-edge from a reachable point w: the
    nearest reachable point among v's own candidates, else among the 64
    sample points nearest v. The edge goes into a free slot of w's row when
    there is one, else replaces w's farthest out-edge whose target has at
    least two in-edges from reachable points (so it stays reachable).
    """
    n, R = adj.shape

    def reach_indeg(seen):
        src = np.repeat(seen, R)
        t = adj.reshape(-1).astype(np.int64)
        ok = src & (adj.reshape(-1) != PAD)
        return np.bincount(t[ok], minlength=n)

    for _ in range(rounds):
        seen = _reachable(n, adj, s_id)
        if seen.all():
            return adj
        indeg = reach_indeg(seen)
        ok_P = P[seen[P]]
        ok_Pf = vectors[ok_P].astype(np.float64)
        for v in np.flatnonzero(~seen):
            if seen[v]:
                continue
            ws = [int(w) for w in cand[v] if w >= 0 and seen[w] and w != v]
            x = vectors[v].astype(np.float64)
            ws += [int(ok_P[i]) for i in np.argsort(((ok_Pf - x) ** 2).sum(1), kind="stable")[:64]
                   if ok_P[i] != v]
            linked = False
            for w in ws:
                row = adj[w]
                pads = np.flatnonzero(row == PAD)
                if pads.size:
                    row[pads[0]] = v
                    linked = True
                    break
            if not linked:
                for w in ws:
                    row = adj[w]
                    movable = [j for j in range(R - 1, -1, -1) if indeg[row[j]] >= 2]
                    if movable:
                        indeg[row[movable[0]]] -= 1
                        row[movable[0]] = v
                        linked = True
                        break
            if not linked:
                continue
            indeg[v] += 1
            stack = [v]
            seen[v] = True
            while stack:
                u = stack.pop()
                for t in adj[u]:
                    if t == PAD:
                        continue
                    indeg[t] += 1
                    if not seen[t]:
                        seen[t] = True
                        stack.append(int(t))
    seen = _reachable(n, adj, s_id)
    if not seen.all():
        raise RuntimeError(f"graph repair left {int((~seen).sum())} unreachable points")
    return adj
