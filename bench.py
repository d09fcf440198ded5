#!/usr/bin/env python3
"""Benchmark of the BOA adaptive filtered search on one MI355X.

One step = one adaptive search (all phases) of the whole query batch of
the workload, with the index, queries and ranges resident in HBM. The
default workload is the largest one-GPU configuration, u8-10M-d128 (10M
uint8 vectors, R = 32). Prints one JSON line: filtered QPS, recall@10
against exhaustive filtered search (every returned id verified on its own:
predicates, repeats, float64 distance recomputed from the vectors), average
final beamwidth, the fixed-width (L=500) baseline built from the same
kernel, the paper's own operating point (eps 0.05, alpha 2), the roofline
position of the search kernel (algorithmic gathered bytes over the
kernel's HIP-event time), the same search with its host transfers inside
the timed loop (queries in, results out; reported beside the value, never
as it), and the CPU oracle timed on the host cores.

The operating point (eps, alpha) is the fastest point of a grid whose
recall reaches the target on a held-out query batch of the same recipe
(other seed parts); QPS and recall are then reported on the evaluation
batch, which played no part in the choice.

The graph is built in-process by the workloads package (exact kNN on the
GPU with torch matmul, then pruning and a navigation layer); that is input
preparation, outside the timed region.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "filtered QPS at recall@10 >= 0.95 (1 GPU); avg beamwidth; HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0
KERNEL = "boa::phase_kernel"


def log(msg: str):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def exact_filtered_topk(torch, X, attrs_t, f32_cols, Q, ranges_t, k, chunk=256):
    """Exhaustive filtered top-k on the GPU (measurement only): squared L2 by
    the norm expansion in float64 from float32 GEMM pieces, predicates per
    column type. Returns ids (nq,k) int64, d (nq,k) float64, n_valid (nq)."""
    n = X.shape[0]
    xn = (X.double() ** 2).sum(1)
    ids_out, d_out, nv_out = [], [], []
    a_i = attrs_t
    a_f = attrs_t.view(torch.float32)
    for s in range(0, Q.shape[0], chunk):
        q = Q[s:s + chunk]
        r = ranges_t[s:s + chunk]
        dot = (q @ X.T).double()
        d = (q.double() ** 2).sum(1)[:, None] + xn[None, :] - 2.0 * dot
        valid = torch.ones((q.shape[0], n), dtype=torch.bool, device=X.device)
        for j in range(attrs_t.shape[1]):
            if j in f32_cols:
                col = a_f[:, j][None, :]
                lo = r[:, j, 0].view(torch.float32)[:, None]
                hi = r[:, j, 1].view(torch.float32)[:, None]
            else:
                col = a_i[:, j][None, :]
                lo = r[:, j, 0][:, None]
                hi = r[:, j, 1][:, None]
            valid &= (lo <= col) & (col <= hi)
        d = torch.where(valid, d, torch.full_like(d, float("inf")))
        # candidates by the expanded form, then exact float64 distances by the
        # direct form (the expansion cancels badly for near points)
        kk = min(n, k + 32)
        dv, di = torch.topk(d, kk, dim=1, largest=False, sorted=True)
        xd = X[di].double() - q.double()[:, None, :]
        de = (xd * xd).sum(-1)
        de = torch.where(torch.isfinite(dv), de, torch.full_like(de, float("inf")))
        o = torch.argsort(di, dim=1, stable=True)
        de, di = de.gather(1, o), di.gather(1, o)
        o = torch.argsort(de, dim=1, stable=True)
        ids_out.append(di.gather(1, o)[:, :k])
        d_out.append(de.gather(1, o)[:, :k])
        nv_out.append(valid.sum(1))
        del dot, d, valid, xd
    return torch.cat(ids_out).cpu().numpy(), torch.cat(d_out).cpu().numpy(), torch.cat(nv_out).cpu().numpy()


def verified_rows(ids, X, Q, attrs, ranges, attr_dtypes):
    """Each returned id checked independently of the search: whether it
    satisfies its query's range predicates (Eq. 2, per column type), and its
    squared distance to the query recomputed in float64 from the vectors.
    Returns (ok: returned, valid, and not a repeat of an earlier id in its
    row; d64: recomputed distances)."""
    from workloads import gen
    ids = ids.astype(np.int64)
    nq, k = ids.shape
    pad = ids == 0xFFFFFFFF
    safe = np.where(pad, 0, ids)
    ok = ~pad
    a = attrs[safe]
    for j, t in enumerate(attr_dtypes):
        lo, hi = ranges[:, j, 0][:, None], ranges[:, j, 1][:, None]
        col = a[:, :, j]
        if t == gen.ATTR_F32:
            col, lo, hi = gen.cells_as_f32(col), gen.cells_as_f32(lo), gen.cells_as_f32(hi)
        ok &= (lo <= col) & (col <= hi)
    for j in range(1, k):   # a repeated id counts once
        ok[:, j] &= ~(safe[:, j:j + 1] == safe[:, :j]).any(1)
    d64 = np.empty((nq, k), dtype=np.float64)
    for s0 in range(0, nq, 1000):
        x = X[safe[s0:s0 + 1000]].astype(np.float64)
        d64[s0:s0 + 1000] = ((x - Q[s0:s0 + 1000].astype(np.float64)[:, None, :]) ** 2).sum(-1)
    return ok, d64


def recall(ids, gt_ids, gt_d, n_valid, k, ver, per_query=False):
    """strict: |returned valid ids ∩ GT| / min(k, |D_f|); tie-tolerant: returned
    valid, distinct ids whose recomputed float64 distance does not exceed the
    k-th exact distance (rel 1e-5). `ver` = verified_rows(...) of `ids`: an id
    that fails its predicates or repeats counts for nothing, and the distance
    the search reported is never used."""
    ok, d64 = ver
    ids = ids.astype(np.int64)
    denom = np.maximum(1, np.minimum(k, n_valid))
    strict = np.zeros(len(ids))
    tie = np.zeros(len(ids))
    for i in range(len(ids)):
        f = ids[i][ok[i]]
        g = gt_ids[i][np.isfinite(gt_d[i])]
        returned = int((ids[i] != 0xFFFFFFFF).sum())
        if len(g):
            strict[i] = len(set(f.tolist()) & set(g.tolist())) / denom[i]
            dk = gt_d[i][len(g) - 1]
            tie[i] = min(k, int((d64[i][ok[i]] <= dk * (1 + 1e-5) + 1e-12).sum())) / denom[i]
        else:   # no valid point: returning nothing is the whole answer
            strict[i] = tie[i] = 1.0 if returned == 0 else 0.0
    if per_query:
        return tie
    return float(strict.mean()), float(tie.mean())


def source_digest() -> str:
    """sha256 over the search library's sources (kernels and launch planning)
    and the workload's input generators (data and graph): a change to any of
    them can change the HBM traffic of a launch."""
    import hashlib
    h = hashlib.sha256()
    for f in ("paper_2609_16175_amd/csrc/boa_kernels.hip", "paper_2609_16175_amd/csrc/boa_api.hip",
              "paper_2609_16175_amd/csrc/boa_internal.h", "workloads/gen.py", "workloads/graph.py"):
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()


def recorded_traffic(workload: str):
    """HBM bytes per launch from the committed counter runs, only while the
    library sources are the ones they measured (else None)."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))[workload]
        if source_digest() != rec["source_sha256"]:
            return None
        return float(rec["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


SEL_EDGES = (0.0, 1e-4, 1e-3, 1e-2, 0.03, 0.1, 0.3, 1.0)


def selectivity_summary(n_valid, n: int, k: int, per_query_recall=None) -> dict:
    """Realised joint selectivity of the query ranges (|D_f| / n per query,
    from the exhaustive pass): quantiles, a histogram over fixed bins, the
    queries with fewer than k valid points, and (given per-query recall)
    the mean recall of each bin."""
    nv = np.asarray(n_valid, dtype=np.int64)
    sel = nv.astype(np.float64) / n
    counts, _ = np.histogram(sel, bins=SEL_EDGES)
    label = [f"{lo:g}-{hi:g}" for lo, hi in zip(SEL_EDGES[:-1], SEL_EDGES[1:])]
    out = {"median": round(float(np.median(sel)), 6), "p5": round(float(np.percentile(sel, 5)), 6),
           "p95": round(float(np.percentile(sel, 95)), 6), "min_valid_points": int(nv.min()),
           "queries_with_fewer_than_k": int((nv < k).sum()),
           "histogram": {lb: int(c) for lb, c in zip(label, counts)}}
    if per_query_recall is not None:
        rq = np.asarray(per_query_recall, dtype=np.float64)
        b = np.clip(np.searchsorted(SEL_EDGES, sel, side="right") - 1, 0, len(label) - 1)
        out["recall_by_bin"] = {label[i]: round(float(rq[b == i].mean()), 4)
                                for i in range(len(label)) if (b == i).any()}
    return out


def cpu_info() -> dict:
    """Host CPU: model name and socket count (lscpu, else /proc/cpuinfo),
    logical CPUs (nproc) and the CPUs this process may run on."""
    import subprocess
    info = {"nproc": os.cpu_count() or 1, "affinity": len(os.sched_getaffinity(0))}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        kv = {l.split(":", 1)[0].strip(): l.split(":", 1)[1].strip() for l in out.splitlines() if ":" in l}
        info["model"] = kv.get("Model name", platform.machine())
        info["sockets"] = int(kv.get("Socket(s)", "1"))
        info["threads_per_core"] = int(kv.get("Thread(s) per core", "1"))
    except (OSError, ValueError, subprocess.SubprocessError):
        try:
            txt = open("/proc/cpuinfo").read()
            names = [l.split(":", 1)[1].strip() for l in txt.splitlines() if l.startswith("model name")]
            info["model"] = names[0] if names else platform.machine()
            info["sockets"] = max(1, len({l for l in txt.splitlines() if l.startswith("physical id")}))
        except OSError:
            info["model"] = platform.machine()
    return info


def doubling_widths(L0: int, Lmax: int) -> list:
    """The widths L0, 2 L0, ... up to Lmax (the alpha = 2 schedule)."""
    out, L = [], L0
    while True:
        out.append(L)
        if L >= Lmax:
            return out
        L = min(2 * L, Lmax)


def gathered_bytes(stats) -> float:
    return float(sum(p["gathered_bytes"] for p in stats["phases"]))


def gathered_bytes_phase(stats, i: int) -> float:
    return float(stats["phases"][i]["gathered_bytes"])


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="u8-10M-d128")
    ap.add_argument("--n", type=int, default=0, help="scale the workload down to n points (testing)")
    ap.add_argument("--nq", type=int, default=0)
    ap.add_argument("--eps", type=float, default=0.0,
                    help="confidence threshold of Eq. 3; 0: choose from --eps-grid (see --alpha)")
    ap.add_argument("--alpha", type=float, default=0.0,
                    help="growth factor of the width schedule; 0: choose from --alpha-grid")
    ap.add_argument("--eps-grid", default="0,0.001,0.005,0.01,0.02,0.05,0.1,0.15,0.2")
    ap.add_argument("--alpha-grid", default="2,32")
    ap.add_argument("--recall-target", type=float, default=0.95)
    ap.add_argument("--fixed-steps", type=int, default=3)
    ap.add_argument("--no-fixed", action="store_true")
    ap.add_argument("--no-lneeded", action="store_true", help="skip the per-query 'L needed' analysis")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle timing")
    ap.add_argument("--lds-slots", type=int, default=0, help="force the LDS visited-table size")
    ap.add_argument("--escalation-waves", type=int, default=0, choices=(0, 1),
                    help="split mode's escalation launch: 0 two waves per query where it applies, 1 one")
    ap.add_argument("--modes", default="phased,fused,split,boa_plus,warm",
                    help="adaptive modes to time (warm: warm-start escalation, fused); the fastest of the "
                         "escalation kind chosen on the held-out batch is the headline")
    ap.add_argument("--no-paper", action="store_true", help="skip the paper's operating point")
    ap.add_argument("--json-out", default="")
    ap.add_argument("--graph-cache", default="", help="npz file: load the graph if present, else save it")
    ap.add_argument("--vector-graph", action="store_true",
                    help="build the graph from vector distances only (no attribute-aware edges)")
    ap.add_argument("--pq", action="store_true",
                    help="traverse with product-quantised distances (4-bit codes, trained offline) and "
                         "re-rank exactly (Alg. 2 PQDist; Sec. III-B)")
    ap.add_argument("--pq-m", type=int, default=0, help="PQ subspaces (default d / 4)")
    ap.add_argument("--copy-probe", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0:
        ap.error("--steps must be >= 1 and --warmup >= 0")

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the search is query-parallel "
                                   "and runs on a single MI355X; multi-GPU query sharding is not built",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import torch
    if args.copy_probe:
        n = args.copy_probe * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda:0")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n * 4, "launches": 3}), flush=True)
        return

    import paper_2609_16175_amd as boa
    from workloads import gen, graph

    wl = gen.BY_NAME[args.workload]
    if args.n:
        wl = wl.scaled(args.n, nq=args.nq or None)
    elif args.nq:
        wl = wl.scaled(wl.n, nq=args.nq, n_clusters=wl.n_clusters)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t = time.time()
    data = gen.generate(wl)
    log(f"generated {wl.name}: n={wl.n} d={wl.d} m={wl.m} nq={wl.nq} in {time.time() - t:.1f}s")
    types = np.array(wl.attr_dtypes, dtype=np.int32)
    t = time.time()
    recipe = f"{wl.name}/n={wl.n}/" + ("vector" if args.vector_graph else "attribute-aware")
    z = np.load(args.graph_cache) if args.graph_cache and os.path.exists(args.graph_cache) else None
    if z is not None and "recipe" in z and str(z["recipe"]) == recipe:
        adj, entry = z["adj"], int(z["entry"])
    else:
        kw = {} if args.vector_graph else dict(attrs=data.attrs, attr_dtypes=types)
        adj, entry = graph.build_graph(data.vectors, wl.R, device=dev, **kw)
        if args.graph_cache:
            np.savez(args.graph_cache, adj=adj, entry=entry, recipe=recipe)
    deg = float((adj != graph.PAD).sum(1).mean())
    log(f"graph R={wl.R} ({recipe}, mean degree {deg:.1f}) entry={entry} in {time.time() - t:.1f}s")
    torch.cuda.empty_cache()

    f32_cols = {j for j, tt in enumerate(wl.attr_dtypes) if tt == gen.ATTR_F32}
    t = time.time()
    # a held-out batch of the same recipe (other seed parts) chooses the
    # operating point; the evaluation batch is only reported on
    ho_q, ho_r, _ = gen.heldout_queries(wl, data, wl.nq)
    Xg = torch.from_numpy(data.vectors).to(dev).float()
    Ag = torch.from_numpy(data.attrs).to(dev)
    chunk = max(8, min(256, (1 << 30) // wl.n))
    gt_ids, gt_d, n_valid = exact_filtered_topk(torch, Xg, Ag, f32_cols, torch.from_numpy(data.queries).to(dev).float(),
                                                torch.from_numpy(data.ranges).to(dev), wl.k, chunk=chunk)
    ho_gt = exact_filtered_topk(torch, Xg, Ag, f32_cols, torch.from_numpy(ho_q).to(dev).float(),
                                torch.from_numpy(ho_r).to(dev), wl.k, chunk=chunk)
    del Xg, Ag
    torch.cuda.empty_cache()
    log(f"exhaustive filtered top-{wl.k} of both batches in {time.time() - t:.1f}s; selectivity median "
        f"{np.median(n_valid) / wl.n:.4f}, min valid {int(n_valid.min())}")

    index = boa.Index(data.vectors, data.attrs, types, adj, entry)
    pq_info = None
    if args.pq:
        from workloads import pq as pqmod
        t = time.time()
        M = args.pq_m or wl.d // 4
        codebook = pqmod.train(data.vectors, M, seed=wl.seed, device=dev)
        codes = pqmod.encode(data.vectors, codebook, device=dev)
        index.set_pq(codebook, codes)
        pq_info = {"subspaces": M, "centroids": 16, "code_bytes": M // 2,
                   "bytes_per_scored_node": M // 2 + 4 * wl.m,
                   "exact_bytes_per_scored_node": wl.d * (1 if wl.vec_dtype == gen.VEC_U8 else 4) + 4 * wl.m}
        log(f"product quantisation: {M} subspaces x 16 centroids, {M // 2} B codes, trained and encoded "
            f"in {time.time() - t:.1f}s")
    q = torch.from_numpy(data.queries).to(dev)
    r = torch.from_numpy(data.ranges).to(dev)
    q_ho = torch.from_numpy(ho_q).to(dev)
    r_ho = torch.from_numpy(ho_r).to(dev)
    base_kw = dict(k=wl.k, L0=wl.L0, Lmax=wl.Lmax, lds_hash_slots=args.lds_slots, pq=args.pq,
                   escalation_waves=args.escalation_waves)

    def timed(search_kw, steps, warmup, qq=q, rr=r):
        """warm-up, then `steps` timed searches bracketed by device syncs;
        per-launch kernel time comes from the library's HIP events."""
        o = None
        for _ in range(warmup):
            o = index.search(qq, rr, **search_kw)
        index.reset_counters()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            o = index.search(qq, rr, **search_kw)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        return (t1 - t0) * 1e3 / steps, index.stats(), o

    def eval_recall(o, heldout=False, per_query=False):
        """recall@k of a search result, every returned id verified (predicates,
        repeats, float64 distance recomputed from the vectors)."""
        ids_o = o.ids.cpu().numpy().view(np.uint32)
        qs, rs = (ho_q, ho_r) if heldout else (data.queries, data.ranges)
        gi, gd, nv = ho_gt if heldout else (gt_ids, gt_d, n_valid)
        ver = verified_rows(ids_o, data.vectors, qs, data.attrs, rs, wl.attr_dtypes)
        return recall(ids_o, gi, gd, nv, wl.k, ver, per_query=per_query)

    # operating point: the metric is QPS at recall@10 >= target, so the
    # confidence threshold eps and the growth factor alpha (inputs of Alg. 1)
    # are chosen on the held-out batch as the fastest grid point that reaches
    # the target there (split mode, a few steps each)
    eps_grid = [args.eps] if args.eps > 0 else [float(x) for x in args.eps_grid.split(",")]
    alpha_grid = [args.alpha] if args.alpha > 0 else [float(x) for x in args.alpha_grid.split(",")]
    # two kinds of escalation: each phase restarting the search (Alg. 1 as
    # printed; timed in split mode here) or continuing from the previous
    # phase's state (warm start, fused mode)
    mode_list = args.modes.split(",")
    kinds = {"restart": {"split": True}, "warm": {"fused": True, "warm": True}}
    if "warm" not in mode_list:
        del kinds["warm"]
    if not [m2 for m2 in mode_list if m2 != "warm"]:
        del kinds["restart"]
    points = [(e, a, kd) for kd in kinds for a in alpha_grid for e in eps_grid]
    sweep = []
    for e, a, kd in points:
        ms_p, st_p, o_p = timed(dict(base_kw, eps=e, alpha=a, **kinds[kd]), 3, 1, q_ho, r_ho)
        fl_p = o_p.final_L.cpu().numpy()
        _, rt_p = eval_recall(o_p, heldout=True)
        sweep.append(dict(eps=e, alpha=a, escalation=kd, schedule=[p["L"] for p in st_p["phases"]],
                          ms_per_step=round(ms_p, 4), qps=round(wl.nq / (ms_p / 1e3), 1),
                          recall_at_10=round(rt_p, 5), L_avg=round(float(fl_p.mean()), 2)))
        log(f"held-out point eps={e} alpha={a} {kd}: {ms_p:.3f} ms/step, recall {rt_p:.4f}, "
            f"L_avg {fl_p.mean():.1f}")

    def choose(pts):
        ok = [p for p in pts if p["recall_at_10"] >= args.recall_target]
        return (min(ok, key=lambda p: p["ms_per_step"]) if ok else max(pts, key=lambda p: p["recall_at_10"])), bool(ok)

    chosen, _ = choose(sweep)
    chosen_kind = {kd: choose([p for p in sweep if p["escalation"] == kd])[0] for kd in kinds}
    log(f"chosen on the held-out batch: eps={chosen['eps']} alpha={chosen['alpha']} {chosen['escalation']} "
        f"({'meets' if chosen['recall_at_10'] >= args.recall_target else 'MISSES'} recall@10 >= "
        f"{args.recall_target} there)")

    # every restart mode at the restart kind's point (identical results), the
    # warm mode at the warm kind's point; the headline is the chosen kind's
    # fastest mode
    mode_kw = {"phased": {}, "fused": {"fused": True}, "split": {"split": True},
               "boa_plus": {"boa_plus": True, "sub_batches": wl.sub_batches},
               "warm": {"fused": True, "warm": True}}
    kw_kind = {kd: dict(base_kw, eps=c["eps"], alpha=c["alpha"]) for kd, c in chosen_kind.items()}
    modes = {}
    for mode in mode_list:
        kd = "warm" if mode == "warm" else "restart"
        ms_m, st_m, out_m = timed(dict(kw_kind[kd], **mode_kw[mode]), args.steps, args.warmup)
        modes[mode] = (ms_m, st_m, out_m)
        log(f"adaptive ({mode}, eps={kw_kind[kd]['eps']} alpha={kw_kind[kd]['alpha']}): {ms_m:.3f} ms/step, "
            f"{wl.nq / (ms_m / 1e3):,.0f} QPS")
    restart_modes = [m2 for m2 in modes if m2 != "warm"]
    if restart_modes:
        ids_r = modes[restart_modes[0]][2].ids.cpu().numpy().view(np.uint32)
        for m2 in restart_modes:
            assert np.array_equal(modes[m2][2].ids.cpu().numpy().view(np.uint32), ids_r), f"{m2} results differ"
    mode = "warm" if chosen["escalation"] == "warm" else min(restart_modes, key=lambda k2: modes[k2][0])
    kw = kw_kind[chosen["escalation"]]
    ms, st, out = modes[mode]
    qps = wl.nq / (ms / 1e3)
    other_kind = None
    other = "restart" if mode == "warm" else "warm"
    if other in kinds:
        om = "warm" if other == "warm" else min(restart_modes, key=lambda k2: modes[k2][0])
        rs_o, rt_o = eval_recall(modes[om][2])
        other_kind = dict(escalation=other, mode=om, eps=kw_kind[other]["eps"], alpha=kw_kind[other]["alpha"],
                          ms_per_step=round(modes[om][0], 4), qps=round(wl.nq / (modes[om][0] / 1e3), 1),
                          recall_at_10=round(rt_o, 5), recall_at_10_strict=round(rs_o, 5),
                          L_avg=round(float(modes[om][2].final_L.cpu().numpy().mean()), 2))

    ids = out.ids.cpu().numpy().view(np.uint32)
    final_L = out.final_L.cpu().numpy()
    rec_strict, rec_tie = eval_recall(out)
    target_met = rec_tie >= args.recall_target
    sched = [p["L"] for p in st["phases"]]
    L_avg = float(final_L.mean())
    L_work = float(sum(p["L"] * p["active"] for p in st["phases"]) / wl.nq)
    split = {str(p["L"]): round(100.0 * float((final_L == p["L"]).mean()), 2) for p in st["phases"]}
    rq = eval_recall(out, per_query=True)
    rec_by_L = {str(p["L"]): round(float(rq[final_L == p["L"]].mean()), 4)
                for p in st["phases"] if (final_L == p["L"]).any()}
    log(f"evaluation batch: recall@10 {rec_tie:.4f} (strict {rec_strict:.4f}); L_avg {L_avg:.1f}; "
        f"split {split}; recall by final L {rec_by_L}")

    # the same search with its host transfers inside the timed loop: queries
    # and ranges copied from pinned host memory to HBM, the results copied
    # back (a caller whose queries arrive over PCIe); not the headline value,
    # which has the inputs resident in HBM
    qh, rh = torch.from_numpy(data.queries).pin_memory(), torch.from_numpy(data.ranges).pin_memory()
    hosts = [torch.empty(t.shape, dtype=t.dtype).pin_memory() for t in (out.ids, out.dists, out.final_L)]
    e2e_kw = dict(kw, **mode_kw[mode])
    for it in range(args.warmup + args.steps):
        if it == args.warmup:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        o_h = index.search(qh.to(dev, non_blocking=True), rh.to(dev, non_blocking=True), **e2e_kw)
        for h, t_dev in zip(hosts, (o_h.ids, o_h.dists, o_h.final_L)):
            h.copy_(t_dev, non_blocking=True)
        torch.cuda.synchronize()
    ms_e2e = (time.perf_counter() - t0) * 1e3 / args.steps
    assert np.array_equal(hosts[0].numpy().view(np.uint32), ids), "end-to-end results differ"
    e2e = dict(mode=mode, ms_per_step=round(ms_e2e, 4), qps=round(wl.nq / (ms_e2e / 1e3), 1),
               host_bytes_per_step=int(qh.numel() * qh.element_size() + rh.numel() * rh.element_size()
                                       + sum(h.numel() * h.element_size() for h in hosts)))
    log(f"end to end with host transfers ({mode}): {ms_e2e:.3f} ms/step, {e2e['qps']:,.0f} QPS")

    # roofline of the dominant kernel: launches are grouped by the phase they
    # start at (a split search has two kernels: the first phase, and the
    # escalation through every later phase); each group's algorithmic bytes
    # are the gathered bytes of the phases its launches cover
    nph = len(st["phases"])
    starts = [i for i in range(nph) if st["cum_phase_launches"][i] > 0]
    groups = []
    for gi, i in enumerate(starts):
        j = starts[gi + 1] if gi + 1 < len(starts) else nph
        if mode in ("fused", "warm"):
            j = nph
        nl = st["cum_phase_launches"][i]
        kms = st["cum_phase_kernel_ms"][i] / nl
        b = sum(gathered_bytes_phase(st, q2) for q2 in range(i, j)) * args.steps / nl
        groups.append(dict(phases=f"{st['phases'][i]['L']}..{st['phases'][j - 1]['L']}", launches=nl,
                           avg_launch_ms=round(kms, 5), bytes_per_launch=round(b),
                           GBps=round(b / (kms * 1e-3) / 1e9, 1),
                           time_share=round(st["cum_phase_kernel_ms"][i] / st["cum_kernel_ms"], 4)))
    dom = max(groups, key=lambda g: g["time_share"])
    bytes_launch, avg_launch_ms = dom["bytes_per_launch"], dom["avg_launch_ms"]
    achieved = dom["GBps"]
    kernel_share = st["cum_kernel_ms"] / (ms * args.steps)
    log(f"kernel ({mode}): dominant launch group {dom['phases']}: {avg_launch_ms:.4f} ms/launch avg over "
        f"{dom['launches']} launches, {bytes_launch / 1e6:.2f} MB/launch -> {achieved:.1f} GB/s; "
        f"kernel time share {kernel_share:.2f}; groups {groups}")

    # "L needed" (the paper's motivation figure): per query, the narrowest
    # width of the alpha = 2 schedule whose fixed-width search already
    # returns its exact filtered top-k; set against the width the adaptive
    # search stopped at, it shows what the confidence test decides well
    # (stopped early enough and right) and badly (stopped too early: lost)
    lneed = None
    if not args.no_lneeded:
        widths = doubling_widths(wl.L0, wl.Lmax)
        need = np.full(wl.nq, np.iinfo(np.int32).max, dtype=np.int64)
        for Lw in reversed(widths):
            o = index.search(q, r, k=wl.k, fixed_L=Lw, pq=args.pq)
            rq_w = eval_recall(o, per_query=True)
            need[rq_w >= 1.0 - 1e-9] = Lw
        lneed = {"widths": widths,
                 "pct_by_L_needed": {str(Lw): round(100.0 * float((need == Lw).mean()), 2) for Lw in widths},
                 "pct_beyond_Lmax": round(100.0 * float((need > wl.Lmax).mean()), 2),
                 "pct_stopped_below_L_needed": round(100.0 * float((final_L < need).mean()), 2),
                 "pct_escalated_past_L_needed": round(100.0 * float((final_L > need).mean()), 2)}
        log(f"L needed: {lneed}")

    def paper_leg(pmode):
        """the paper's own point (eps 0.05, alpha 2; Sec. IV) on the
        evaluation batch, restarting (in pmode) and with warm start"""
        msp, stp, out_p = timed(dict(base_kw, eps=0.05, alpha=2.0, **mode_kw[pmode]), args.fixed_steps, 1)
        rps, rpt = eval_recall(out_p)
        paper_point = dict(eps=0.05, alpha=2.0, mode=pmode, schedule=[p["L"] for p in stp["phases"]],
                           ms_per_step=round(msp, 4), qps=round(wl.nq / (msp / 1e3), 1), recall_at_10=round(rpt, 5),
                           recall_at_10_strict=round(rps, 5),
                           L_avg=round(float(out_p.final_L.cpu().numpy().mean()), 2),
                           speedup_vs_fixed_L500=round((wl.nq / (msp / 1e3)) / fixed["qps"], 3)
                           if fixed else None)
        log(f"paper's point eps=0.05 alpha=2 ({pmode}): {msp:.3f} ms/step, recall {rpt:.4f}")
        # the same point with warm-start escalation
        msw, _, out_w = timed(dict(base_kw, eps=0.05, alpha=2.0, **mode_kw["warm"]), args.fixed_steps, 1)
        _, rwt = eval_recall(out_w)
        paper_point["warm"] = dict(ms_per_step=round(msw, 4), qps=round(wl.nq / (msw / 1e3), 1),
                                   recall_at_10=round(rwt, 5),
                                   L_avg=round(float(out_w.final_L.cpu().numpy().mean()), 2),
                                   speedup_vs_fixed_L500=round((wl.nq / (msw / 1e3)) / fixed["qps"], 3) if fixed else None)
        log(f"paper's point with warm start: {msw:.3f} ms/step, recall {rwt:.4f}")
        return paper_point

    fixed = None
    if not args.no_fixed:
        msf, stf, out_f = timed(dict(k=wl.k, fixed_L=500, pq=args.pq), args.fixed_steps, 1)
        rs, rt = eval_recall(out_f)
        fixed = dict(L=500, ms_per_step=round(msf, 4), qps=round(wl.nq / (msf / 1e3), 1),
                     recall_at_10=round(rt, 5), recall_at_10_strict=round(rs, 5),
                     gathered_GBps=round(gathered_bytes(stf) / (stf["phases"][0]["kernel_ms"] * 1e-3) / 1e9, 1))
        log(f"fixed L=500: {msf:.3f} ms/step, {fixed['qps']:,.0f} QPS, recall {rt:.4f}")

    # the paper's own point (eps 0.05, alpha 2; Sec. IV), on the evaluation
    # batch, in the fastest mode
    paper_point = None
    if not args.no_paper:
        pmode = min(restart_modes, key=lambda k2: modes[k2][0]) if restart_modes else "split"
        paper_point = paper_leg(pmode)


    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        ci = cpu_info()
        # the CPUs this process may run on (the GPU machine gives each GPU a share
        # of the host; nproc counts the whole host), at most 16
        threads = max(1, min(16, ci["affinity"]))
        oix = oracle.Index(data.vectors, data.attrs, types, adj, entry,
                           *((codebook, codes) if args.pq else (None, None)))
        osched = oracle.schedule(wl.L0, chosen["alpha"], wl.Lmax)

        def run_oracle(n_q, nt):
            """the oracle of the chosen escalation on the first n_q queries,
            nt threads over independent queries"""
            if chosen["escalation"] != "warm":
                return oracle.boa(oix, data.queries[:n_q], data.ranges[:n_q], wl.k, osched, eps=chosen["eps"],
                                  threads=nt)
            from concurrent.futures import ThreadPoolExecutor
            cuts = np.linspace(0, n_q, nt + 1).astype(int)
            with ThreadPoolExecutor(nt) as ex:
                parts = list(ex.map(lambda ab: oracle.boa_warm(oix, data.queries[ab[0]:ab[1]],
                                                               data.ranges[ab[0]:ab[1]], wl.k, osched,
                                                               eps=chosen["eps"]),
                                    [(a, b) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]))
            return type(parts[0])(np.concatenate([p_.ids for p_ in parts]),
                                  np.concatenate([p_.dists for p_ in parts]),
                                  np.concatenate([p_.final_L for p_ in parts]),
                                  np.concatenate([p_.expansions for p_ in parts]),
                                  np.concatenate([p_.scored for p_ in parts]), [])

        # calibrate, then size the sample to the time budget
        n0 = min(wl.nq, 4 * threads)
        tc = time.perf_counter()
        run_oracle(n0, threads)
        per_q = (time.perf_counter() - tc) / n0
        ns = int(min(wl.nq, max(n0, args.cpu_seconds / max(per_q, 1e-6))))
        tc = time.perf_counter()
        ref = run_oracle(ns, threads)
        el = time.perf_counter() - tc
        same = int(((ref.ids == ids[:ns]).all(1) & (ref.final_L == final_L[:ns])).sum())
        # the oracle on one thread as well (a smaller sample of the same queries)
        n1 = int(min(ns, max(1, (args.cpu_seconds / 3.0) / max(el * threads / ns, 1e-6))))
        tc = time.perf_counter()
        run_oracle(n1, 1)
        el1 = time.perf_counter() - tc
        cpu = dict(value=round(ns / el, 2), unit="queries/s", cores=threads, kind="oracle",
                   sample=f"first {ns} of {wl.nq} queries, full adaptive schedule "
                          f"({chosen['escalation']} escalation), {threads} threads, "
                          f"{el:.1f}s wall",
                   one_thread_value=round(n1 / el1, 2), one_thread_sample=f"first {n1} queries, {el1:.1f}s wall",
                   cpu_model=ci.get("model"), sockets=ci.get("sockets"), nproc=ci["nproc"],
                   cpus_available=ci["affinity"],
                   gpu_identical_on_sample=f"{same}/{ns}")
        log(f"cpu oracle: {cpu['value']:.1f} QPS on {ns} queries x {threads} threads "
            f"({ci.get('model')}, {ci.get('sockets')} socket(s), nproc {ci['nproc']}); GPU identical on {same}/{ns}")

    res = {
        "metric": METRIC,
        "value": round(qps, 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if wl.vec_dtype == gen.VEC_F32 else "u8",
        "data": "synthetic",
        "config": {"workload": wl.name, "n": wl.n, "d": wl.d, "R": wl.R, "m": wl.m, "nq": wl.nq,
                   "distance": "product-quantised traversal, exact re-rank" if args.pq else "exact",
                   "k": wl.k, "L0": wl.L0, "Lmax": wl.Lmax, "alpha": chosen["alpha"], "eps": chosen["eps"],
                   "schedule": sched, "escalation": chosen["escalation"],
                   "mode": f"BOA ({mode} phases)" if mode != "warm" else "BOA (warm-start escalation, fused)",
                   "graph": recipe,
                   "operating_point_chosen_on": "held-out batch of the same recipe"},
        "modes": {m2: {"ms_per_step": round(v[0], 4), "qps": round(wl.nq / (v[0] / 1e3), 1),
                       "launches_per_step": round(v[1]["cum_launches"] / max(1, v[1]["cum_searches"]), 2)}
                  for m2, v in modes.items()},
        "recall_at_10": round(rec_tie, 5),
        "recall_at_10_strict": round(rec_strict, 5),
        "L_avg": round(L_avg, 2),
        "L_work": round(L_work, 2),
        "phase_split_pct": split,
        "recall_by_final_L": rec_by_L,
        "selectivity": selectivity_summary(n_valid, wl.n, wl.k, rq),
        "phases": [{k2: (round(v, 4) if isinstance(v, float) else v) for k2, v in p.items()}
                   for p in st["phases"]],
        "L_needed": lneed,
        "recall_target": args.recall_target,
        "recall_target_met": bool(target_met),
        "operating_points_heldout": sweep,
        "other_escalation": other_kind,
        "paper_point": paper_point,
        "fixed_L500": fixed,
        "speedup_vs_fixed_L500": round(qps / fixed["qps"], 3) if fixed else None,
        "gathered_GBps_whole_search": round(gathered_bytes(st) * args.steps / (st["cum_kernel_ms"] * 1e-3) / 1e9, 1),
        "end_to_end_with_host_transfers": e2e,
        "roofline": {"bound": "hbm", "kernel": KERNEL, "mode": mode, "phases": dom["phases"],
                     "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic(f"{wl.name}/{mode}/{dom['phases']}"),
                     "bytes_per_launch": round(bytes_launch),
                     "avg_launch_ms": round(avg_launch_ms, 5), "launches": dom["launches"],
                     "launch_groups": groups},
        "cpu_baseline": cpu,
        "product_quantisation": pq_info,
    }
    line = json.dumps(res)
    print(line, flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")


if __name__ == "__main__":
    main()
