"""Seeded synthetic workloads: shapes, value ranges and predicate selectivity.

Each workload is generated scaled down (fewer points and queries, same
recipe) and checked against the configuration it stands for: vector type and
value range, attribute domains, and the joint selectivity of the query
ranges, measured by brute force on the generated attributes.
"""
import dataclasses

import numpy as np
import pytest

from workloads import gen

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

N_SMALL, NQ_SMALL = 20_000, 200


def small(wl):
    return dataclasses.replace(wl, n=min(wl.n, N_SMALL), nq=NQ_SMALL)


@pytest.fixture(scope="module")
def datasets():
    return {wl.name: gen.generate(small(wl)) for wl in gen.WORKLOADS}


def valid_fraction(data, q):
    """Share of the points that satisfy every range predicate of query q."""
    wl = data.wl
    ok = np.ones(wl.n, dtype=bool)
    for j in range(wl.m):
        lo, hi = data.ranges[q, j]
        col = data.attrs[:, j]
        if wl.attr_dtypes[j] == gen.ATTR_F32:
            col = gen.cells_as_f32(col)
            lo, hi = gen.cells_as_f32(np.array([lo, hi], dtype=np.int32))
        ok &= (col >= lo) & (col <= hi)
    return ok.mean()


@pytest.mark.parametrize("wl", gen.WORKLOADS, ids=lambda w: w.name)
def test_shapes_types_and_determinism(wl, datasets):
    d = datasets[wl.name]
    w = d.wl
    assert d.vectors.shape == (w.n, w.d) and d.queries.shape == (w.nq, w.d)
    want = np.uint8 if w.vec_dtype == gen.VEC_U8 else np.float32
    assert d.vectors.dtype == want and d.queries.dtype == want
    assert d.attrs.shape == (w.n, w.m) and d.attrs.dtype == np.int32
    assert d.ranges.shape == (w.nq, w.m, 2) and d.ranges.dtype == np.int32
    assert len(w.attr_dtypes) == w.m
    again = gen.generate(w)
    for a, b in ((d.vectors, again.vectors), (d.attrs, again.attrs),
                 (d.queries, again.queries), (d.ranges, again.ranges)):
        assert np.array_equal(a, b)


def test_vector_value_ranges(datasets):
    sift = datasets["sift-like-1M-d128"]
    v = sift.vectors
    assert np.array_equal(v, np.rint(v)) and v.min() >= 0 and v.max() <= 255
    for name in ("deep-like-1M-d96", "dblp-like-1M-d768"):
        for x in (datasets[name].vectors, datasets[name].queries):
            assert np.abs(np.linalg.norm(x.astype(np.float64), axis=1) - 1.0).max() < 1e-5
    u8 = datasets["u8-10M-d128"].vectors
    assert u8.dtype == np.uint8 and u8.max() > 200 and u8.min() < 50


def test_ranges_are_ordered(datasets):
    for d in datasets.values():
        for j in range(d.wl.m):
            lo, hi = d.ranges[:, j, 0], d.ranges[:, j, 1]
            if d.wl.attr_dtypes[j] == gen.ATTR_F32:
                lo, hi = gen.cells_as_f32(lo), gen.cells_as_f32(hi)
            assert np.all(lo <= hi)


def test_joint_selectivity(datasets):
    sel = {name: np.array([valid_fraction(d, q) for q in range(d.wl.nq)])
           for name, d in datasets.items()}
    # tiny: one range of about half the domain
    assert np.all(np.abs(sel["tiny-10k-d32"] - 0.5) < 0.03)
    # sift-like: each query's joint selectivity is one of 50%, 10%, 1%,
    # drawn uniformly
    s = sel["sift-like-1M-d128"]
    levels = np.array([0.5, 0.1, 0.01])
    nearest = np.argmin(np.abs(np.log(s[:, None] / levels[None, :])), axis=1)
    assert np.all(np.abs(s / levels[nearest] - 1.0) < 0.35)
    share = np.bincount(nearest, minlength=3) / s.size
    assert np.all(share > 0.2)
    # deep-like about 5%, u8 about 10%, dblp-like about 1%
    assert 0.04 < np.median(sel["deep-like-1M-d96"]) < 0.07
    assert np.all(np.abs(sel["u8-10M-d128"] - 0.1) < 0.01)
    assert 0.005 < np.median(sel["dblp-like-1M-d768"]) < 0.03
    assert sel["dblp-like-1M-d768"].min() > 0


def test_attribute_domains(datasets):
    deep = datasets["deep-like-1M-d96"].attrs
    assert deep[:, 0].min() >= 0 and deep[:, 0].max() < 10_000
    z = deep[:, 1]
    assert z.min() >= 0 and z.max() < 1000
    # Zipf(1.1) over 1,000 values: P(0) = 1 / sum_i (i+1)^-1.1
    p0 = 1.0 / np.sum((np.arange(1000) + 1.0) ** -1.1)
    assert abs(np.mean(z == 0) - p0) < 0.02
    f = gen.cells_as_f32(deep[:, 2])
    assert f.min() >= 0.0 and f.max() < 1.0
    sift = datasets["sift-like-1M-d128"].attrs
    assert sift.min() >= 0 and sift.max() < 10_000
    u8 = datasets["u8-10M-d128"].attrs
    assert u8.min() >= 0 and u8.max() < 100_000


def test_dblp_cluster_attributes_and_windows():
    w = small(gen.DBLPLIKE)
    d = gen.generate(w)
    _, cid = gen._mixture_rows(w, gen._centres(w), w.n, part=2)
    for j in (0, 1):
        off = d.attrs[:, j] - cid
        assert off.min() >= 0 and off.max() < 100
    # every query's window on the two cluster attributes holds all values of
    # its own cluster
    qc = d.query_cluster
    for j in (0, 1):
        assert np.all(d.ranges[:, j, 0] <= qc) and np.all(qc + 99 <= d.ranges[:, j, 1])
        assert np.all(d.ranges[:, j, 1] - d.ranges[:, j, 0] == 299)


@pytest.mark.parametrize("wl", [gen.SIFTLIKE, gen.DEEPLIKE, gen.DBLPLIKE], ids=lambda w: w.name)
def test_low_intrinsic_dimension(wl):
    """Cluster centres span LATENT dimensions; each cluster's noise lies
    mostly on its LOCAL orthonormal directions."""
    c = gen._centres(wl)
    c = c - (128.0 if wl.kind in ("sift", "u8") else 0.0)
    sv = np.linalg.svd(c, compute_uv=False)
    assert sv[gen.LATENT - 1] > 1e3 * sv[gen.LATENT]
    u = gen._local_bases(dataclasses.replace(wl, n_clusters=4))
    for b in u:
        assert np.allclose(b @ b.T, np.eye(gen.LOCAL), atol=1e-12)
