"""Seeded synthetic inputs for filtered graph search.

This module only draws numbers: base vectors, attribute records, query
vectors and per-query range predicates. It holds none of the search
method's arithmetic (no distances, no predicates, no beam logic), so that
both the CPU oracle and the GPU path can take their inputs from here
without sharing any code with each other.

The paper's datasets (SIFT1M, Deep1M, DBLP, YouTube; Sec. IV, Table
"Details of Datasets") are not available, so each workload is a Gaussian
mixture with the dimension, size, attribute count and selectivity mix of
the data it stands in for. The paper draws per-attribute range
selectivity between 1% and 100% (Sec. IV); the workloads below fix the
joint selectivity per workload instead.

Descriptor and embedding data of that kind has a low intrinsic
dimension: its points lie near a low-dimensional structure of the
ambient space, both between clusters and inside them. The 1M- and
10M-point mixtures reproduce that: cluster centres lie in a random
8-dimensional subspace, and 99% of each cluster's noise variance lies on
8 random directions of its own (1% is isotropic). The per-dimension
variances are those of the isotropic recipe (centre spread and sigma),
only their distribution over directions changes. An isotropic mixture
in 96-768 dimensions instead puts every cluster at the same distance
from every other and every point of a cluster at the same distance
from a query, which no real descriptor set does. The tiny workload keeps
its isotropic recipe.

Encoding conventions shared with every consumer:
  * vectors: row-major n x d, float32 or uint8.
  * attributes: row-major n x m cells of 4 bytes, held in an int32 array;
    a float32 column stores its IEEE bit pattern in the int32 cell.
  * ranges: row-major nq x m x 2 cells [lo, hi] (inclusive), same
    per-column encoding as the attributes.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass

import numpy as np

ATTR_I32 = 0
ATTR_F32 = 1
VEC_F32 = 0
VEC_U8 = 1

_CHUNK = 1 << 17  # rows generated per chunk (bounds float64 temporaries)


@dataclass(frozen=True)
class Workload:
    """One synthetic filtered-search workload (sizes and distributions)."""

    name: str
    n: int
    d: int
    vec_dtype: int           # VEC_F32 or VEC_U8
    n_clusters: int
    R: int                   # graph out-degree bound
    m: int                   # attributes per point
    attr_dtypes: tuple       # ATTR_I32 / ATTR_F32 per attribute
    nq: int
    k: int
    L0: int
    Lmax: int
    kind: str                # generator recipe, see _GEN
    seed: int
    boa_plus: bool = False
    sub_batches: int = 10

    def scaled(self, n: int, nq: int | None = None, n_clusters: int | None = None):
        """Same recipe at a smaller size (for CPU tests)."""
        nc = n_clusters if n_clusters is not None else max(2, self.n_clusters * n // self.n)
        return dataclasses.replace(self, n=n, nq=self.nq if nq is None else nq,
                                   n_clusters=nc, name=f"{self.name}@{n}")


@dataclass
class Data:
    wl: Workload
    vectors: np.ndarray      # n x d, float32 or uint8
    attrs: np.ndarray        # n x m int32 cells
    queries: np.ndarray      # nq x d
    ranges: np.ndarray       # nq x m x 2 int32 cells
    query_cluster: np.ndarray  # nq, generating cluster of each query (diagnostics only)


# ---------------------------------------------------------------------------
# Workload table. Sizes follow the five target workloads; seeds are
# 0xB0A00000 + index.

TINY = Workload("tiny-10k-d32", n=10_000, d=32, vec_dtype=VEC_F32, n_clusters=16, R=16,
                m=1, attr_dtypes=(ATTR_I32,), nq=100, k=10, L0=16, Lmax=128,
                kind="tiny", seed=0xB0A00000)
SIFTLIKE = Workload("sift-like-1M-d128", n=1_000_000, d=128, vec_dtype=VEC_F32,
                    n_clusters=1000, R=64, m=2, attr_dtypes=(ATTR_I32, ATTR_I32),
                    nq=10_000, k=10, L0=16, Lmax=512, kind="sift", seed=0xB0A00001)
DEEPLIKE = Workload("deep-like-1M-d96", n=1_000_000, d=96, vec_dtype=VEC_F32,
                    n_clusters=1000, R=64, m=3, attr_dtypes=(ATTR_I32, ATTR_I32, ATTR_F32),
                    nq=10_000, k=10, L0=16, Lmax=512, kind="deep", seed=0xB0A00002)
U8LIKE = Workload("u8-10M-d128", n=10_000_000, d=128, vec_dtype=VEC_U8,
                  n_clusters=10_000, R=32, m=2, attr_dtypes=(ATTR_I32, ATTR_I32),
                  nq=10_000, k=10, L0=16, Lmax=512, kind="u8", seed=0xB0A00003)
DBLPLIKE = Workload("dblp-like-1M-d768", n=1_000_000, d=768, vec_dtype=VEC_F32,
                    n_clusters=2000, R=48, m=4, attr_dtypes=(ATTR_I32,) * 4,
                    nq=10_000, k=10, L0=16, Lmax=1024, kind="dblp", seed=0xB0A00004,
                    boa_plus=True, sub_batches=10)

WORKLOADS = [TINY, SIFTLIKE, DEEPLIKE, U8LIKE, DBLPLIKE]
BY_NAME = {w.name: w for w in WORKLOADS}


def _rng(seed: int, part: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, part])))


def f32_bits(a) -> np.ndarray:
    """float32 values -> their int32 bit patterns (attribute/range cell encoding)."""
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32)).view(np.int32)


def cells_as_f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32)).view(np.float32)


# ---------------------------------------------------------------------------
# vector mixtures

LATENT = 8          # dimension of the subspace holding the cluster centres
LOCAL = 8           # directions carrying a cluster's noise
LOCAL_SHARE = 0.99  # share of the noise variance on those directions


def _centres(wl: Workload) -> np.ndarray:
    g = _rng(wl.seed, 1)
    if wl.kind == "tiny":
        return g.normal(0.0, 1.0, size=(wl.n_clusters, wl.d))
    # centres in a random LATENT-dimensional subspace, per-dimension variance
    # 1 on average (40^2 around 128 for the 0..255 workloads)
    basis, _ = np.linalg.qr(g.normal(size=(wl.d, LATENT)))
    z = g.normal(size=(wl.n_clusters, LATENT)) * np.sqrt(wl.d / LATENT)
    c = z @ basis.T
    if wl.kind in ("sift", "u8"):
        return 128.0 + 40.0 * c
    return c


def _local_bases(wl: Workload) -> np.ndarray:
    """n_clusters x LOCAL x d: orthonormal noise directions of each cluster."""
    g = _rng(wl.seed, 6)
    q, _ = np.linalg.qr(g.normal(size=(wl.n_clusters, wl.d, LOCAL)))
    return np.ascontiguousarray(q.transpose(0, 2, 1))


_SIGMA = {"sift": 20.0, "u8": 20.0, "deep": 0.2, "dblp": 0.2}


def _mixture_rows(wl: Workload, centres: np.ndarray, n: int, part: int):
    """n rows of the workload's mixture; returns (rows, cluster_id)."""
    g = _rng(wl.seed, part)
    cid = g.integers(0, wl.n_clusters, size=n)
    out = np.empty((n, wl.d), dtype=np.uint8 if wl.vec_dtype == VEC_U8 else np.float32)
    if wl.kind == "tiny":
        for s in range(0, n, _CHUNK):
            e = min(n, s + _CHUNK)
            c = centres[cid[s:e]]
            out[s:e] = (c + 0.3 * g.standard_normal(size=c.shape)).astype(np.float32)
        return out, cid
    if wl.kind not in _SIGMA:
        raise ValueError(wl.kind)
    U = _local_bases(wl)
    sigma = _SIGMA[wl.kind]
    a_loc = np.sqrt(LOCAL_SHARE * wl.d / LOCAL)
    a_iso = np.sqrt(1.0 - LOCAL_SHARE)
    step = max(4096, (1 << 24) // wl.d)
    for s in range(0, n, step):
        e = min(n, s + step)
        cc = cid[s:e]
        zl = a_loc * g.standard_normal(size=(e - s, LOCAL))
        x = a_iso * g.standard_normal(size=(e - s, wl.d))
        # each cluster's rows get their local directions (one small product
        # per cluster present in the chunk)
        order = np.argsort(cc, kind="stable")
        cs = cc[order]
        cuts = np.flatnonzero(cs[1:] != cs[:-1]) + 1
        for rows in np.split(order, cuts):
            x[rows] += zl[rows] @ U[cc[rows[0]]]
        x = centres[cc] + sigma * x
        if wl.kind in ("sift", "u8"):
            out[s:e] = np.clip(np.rint(x), 0, 255).astype(out.dtype)
        else:
            x /= np.linalg.norm(x, axis=1, keepdims=True)
            out[s:e] = x.astype(np.float32)
    return out, cid


# ---------------------------------------------------------------------------
# attributes and ranges

def _zipf_values(g: np.random.Generator, n: int, domain: int, s: float) -> np.ndarray:
    p = (np.arange(domain, dtype=np.float64) + 1.0) ** (-s)
    cdf = np.cumsum(p / p.sum())
    cdf[-1] = 1.0
    return np.searchsorted(cdf, g.random(n), side="right").astype(np.int32)


def _attributes(wl: Workload, cid: np.ndarray) -> np.ndarray:
    g = _rng(wl.seed, 3)
    n = wl.n
    a = np.empty((n, wl.m), dtype=np.int32)
    if wl.kind == "tiny":
        a[:, 0] = g.integers(0, 1000, size=n)
    elif wl.kind == "sift":
        a[:, 0] = g.integers(0, 10_000, size=n)
        a[:, 1] = g.integers(0, 10_000, size=n)
    elif wl.kind == "u8":
        a[:, 0] = g.integers(0, 100_000, size=n)
        a[:, 1] = g.integers(0, 100_000, size=n)
    elif wl.kind == "deep":
        a[:, 0] = g.integers(0, 10_000, size=n)
        a[:, 1] = _zipf_values(g, n, 1000, 1.1)
        a[:, 2] = f32_bits(g.random(n, dtype=np.float32))
    elif wl.kind == "dblp":
        a[:, 0] = cid + g.integers(0, 100, size=n)
        a[:, 1] = cid + g.integers(0, 100, size=n)
        a[:, 2] = g.integers(0, 10_000, size=n)
        a[:, 3] = g.integers(0, 10_000, size=n)
    else:
        raise ValueError(wl.kind)
    return a


def _uniform_window(g, nq: int, domain: int, width: np.ndarray) -> np.ndarray:
    lo = (g.random(nq) * (domain - width + 1)).astype(np.int64)
    return np.stack([lo, lo + width - 1], axis=1).astype(np.int32)


def _quantile_window(g, nq: int, column_sorted: np.ndarray, frac: float) -> np.ndarray:
    """[lo, hi] covering about `frac` of the column's empirical distribution."""
    n = column_sorted.shape[0]
    u = g.random(nq) * (1.0 - frac)
    i0 = np.floor(u * n).astype(np.int64)
    i1 = np.minimum(n - 1, np.ceil((u + frac) * n).astype(np.int64) - 1)
    return np.stack([column_sorted[i0], column_sorted[i1]], axis=1)


def _ranges(wl: Workload, attrs: np.ndarray, nq: int, qcid: np.ndarray, part: int = 5) -> np.ndarray:
    g = _rng(wl.seed, part)
    r = np.empty((nq, wl.m, 2), dtype=np.int32)
    if wl.kind == "tiny":
        r[:, 0, :] = _uniform_window(g, nq, 1000, np.full(nq, 500))
    elif wl.kind == "sift":
        sel = np.array([0.5, 0.1, 0.01])[g.integers(0, 3, size=nq)]
        w = np.rint(np.sqrt(sel) * 10_000).astype(np.int64)
        r[:, 0, :] = _uniform_window(g, nq, 10_000, w)
        r[:, 1, :] = _uniform_window(g, nq, 10_000, w)
    elif wl.kind == "u8":
        w = np.full(nq, int(round(np.sqrt(0.1) * 100_000)))
        r[:, 0, :] = _uniform_window(g, nq, 100_000, w)
        r[:, 1, :] = _uniform_window(g, nq, 100_000, w)
    elif wl.kind == "deep":
        frac = 0.05 ** (1.0 / 3.0)
        r[:, 0, :] = _quantile_window(g, nq, np.sort(attrs[:, 0]), frac)
        r[:, 1, :] = _quantile_window(g, nq, np.sort(attrs[:, 1]), frac)
        col = np.sort(cells_as_f32(attrs[:, 2]))
        r[:, 2, :] = f32_bits(_quantile_window(g, nq, col, frac))
    elif wl.kind == "dblp":
        # the two cluster-derived attributes get a window of 300 cluster ids
        # placed so that it holds the query's own cluster's values (cluster
        # id + 0..99): the predicate is correlated with where the query lies
        c0 = np.clip(qcid - g.integers(0, 201, size=nq), 0, max(0, wl.n_clusters - 200))
        for j in (0, 1):
            r[:, j, 0] = c0
            r[:, j, 1] = c0 + 299
        w = np.full(nq, int(round(np.sqrt(0.1) * 10_000)))
        r[:, 2, :] = _uniform_window(g, nq, 10_000, w)
        r[:, 3, :] = _uniform_window(g, nq, 10_000, w)
    else:
        raise ValueError(wl.kind)
    return r


def generate(wl: Workload) -> Data:
    """All inputs of one workload, bit-reproducible for a given numpy."""
    centres = _centres(wl)
    vectors, cid = _mixture_rows(wl, centres, wl.n, part=2)
    attrs = _attributes(wl, cid)
    queries, qcid = _mixture_rows(wl, centres, wl.nq, part=4)
    ranges = _ranges(wl, attrs, wl.nq, qcid)
    return Data(wl, vectors, attrs, queries, ranges, qcid)


def heldout_queries(wl: Workload, data: Data, nq: int):
    """A second query batch of the same recipe (other seed parts): queries,
    ranges and generating clusters of `nq` fresh draws. Used to choose
    search parameters without looking at the batch they are reported on."""
    centres = _centres(wl)
    queries, qcid = _mixture_rows(wl, centres, nq, part=7)
    ranges = _ranges(wl, data.attrs, nq, qcid, part=8)
    return queries, ranges, qcid
