"""CPU oracle for BOA filtered beam search — TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. The product library never links it and shares no
code with it. The arithmetic lives in `boa_oracle.c` (plain C, one query
at a time); this module builds it with gcc and marshals numpy arrays.

Inputs use the encoding of `workloads.gen`: vectors n x d (float32 or
uint8), attribute and range cells as int32 (float32 columns hold their
bit patterns), adjacency n x R uint32 padded with 0xFFFFFFFF.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "boa_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
PAD = 0xFFFFFFFF
CFLAGS = ["-O2", "-mfma", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-pthread"]


def build(force: bool = False) -> str:
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, LIB)
    return LIB


class _Index(C.Structure):
    _fields_ = [("n", C.c_int64), ("d", C.c_int32), ("vec_dtype", C.c_int32),
                ("vectors", C.c_void_p), ("m", C.c_int32), ("attrs", C.c_void_p),
                ("attr_dtypes", C.c_void_p), ("R", C.c_int32), ("adj", C.c_void_p),
                ("entry", C.c_int64), ("pq_m", C.c_int32), ("pq_cb", C.c_void_p),
                ("pq_codes", C.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = C.CDLL(LIB)
        P = C.c_void_p
        L.orc_dist_f32.restype = C.c_float
        L.orc_dist_f32.argtypes = [P, P, C.c_int32]
        L.orc_dist_u8.restype = C.c_float
        L.orc_dist_u8.argtypes = [P, P, C.c_int32]
        L.orc_pq_table.restype = None
        L.orc_pq_table.argtypes = [C.POINTER(_Index), P, P]
        L.orc_pq_dist.restype = C.c_float
        L.orc_pq_dist.argtypes = [P, P, C.c_int32]
        L.orc_phi.restype = C.c_int32
        L.orc_phi.argtypes = [P, P, P, C.c_int32]
        L.orc_confident.restype = C.c_int
        L.orc_confident.argtypes = [P, C.c_int32, C.c_int32, C.c_double]
        L.orc_schedule.restype = C.c_int32
        L.orc_schedule.argtypes = [C.c_int32, C.c_double, C.c_int32, P, C.c_int32]
        L.orc_boa.restype = C.c_int32
        L.orc_boa.argtypes = [C.POINTER(_Index), P, P, C.c_int64, C.c_int32, P, C.c_int32,
                              C.c_double, C.c_double, P, P, P, P, P, P, C.c_int32]
        L.orc_boa_warm.restype = C.c_int32
        L.orc_boa_warm.argtypes = [C.POINTER(_Index), P, P, C.c_int64, C.c_int32, P, C.c_int32,
                                   C.c_double, P, P, P, P, P, P]
        L.orc_search_lists.restype = C.c_int32
        L.orc_search_lists.argtypes = [C.POINTER(_Index), P, P, C.c_int64, C.c_int32,
                                       P, P, P, P, P, P]
        L.orc_bruteforce.restype = C.c_int32
        L.orc_bruteforce.argtypes = [C.POINTER(_Index), P, P, C.c_int64, C.c_int32, P, P, P]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


@dataclass
class Index:
    """Host-side view of a graph index for the oracle (keeps arrays alive).
    pq_codebook (M x 16 x d/M float32) and pq_codes (n x M/2 uint8, see
    workloads.pq): traverse with product-quantised distances and re-rank
    the results exactly."""
    vectors: np.ndarray
    attrs: np.ndarray
    attr_dtypes: np.ndarray
    adj: np.ndarray
    entry: int
    pq_codebook: np.ndarray = None
    pq_codes: np.ndarray = None

    def __post_init__(self):
        self.vectors = np.ascontiguousarray(self.vectors)
        assert self.vectors.dtype in (np.float32, np.uint8)
        self.attrs = np.ascontiguousarray(self.attrs, dtype=np.int32)
        self.attr_dtypes = np.ascontiguousarray(self.attr_dtypes, dtype=np.int32)
        self.adj = np.ascontiguousarray(self.adj, dtype=np.uint32)
        n, d = self.vectors.shape
        assert d % 4 == 0
        assert self.attrs.shape == (n, self.attr_dtypes.shape[0])
        assert self.adj.shape[0] == n
        pq_m, cb_p, codes_p = 0, None, None
        if self.pq_codebook is not None:
            self.pq_codebook = np.ascontiguousarray(self.pq_codebook, dtype=np.float32)
            self.pq_codes = np.ascontiguousarray(self.pq_codes, dtype=np.uint8)
            pq_m = self.pq_codebook.shape[0]
            assert self.pq_codebook.shape == (pq_m, 16, d // pq_m) and d % pq_m == 0 and pq_m % 2 == 0
            assert self.pq_codes.shape == (n, pq_m // 2)
            cb_p, codes_p = _p(self.pq_codebook).value, _p(self.pq_codes).value
        self._c = _Index(n, d, 1 if self.vectors.dtype == np.uint8 else 0, _p(self.vectors).value,
                         self.attr_dtypes.shape[0], _p(self.attrs).value,
                         _p(self.attr_dtypes).value, self.adj.shape[1], _p(self.adj).value,
                         int(self.entry), pq_m, cb_p, codes_p)

    @property
    def n(self):
        return self.vectors.shape[0]

    @property
    def m(self):
        return self.attr_dtypes.shape[0]

    def _q(self, queries, ranges):
        q = np.ascontiguousarray(queries, dtype=self.vectors.dtype)
        r = np.ascontiguousarray(ranges, dtype=np.int32)
        assert q.ndim == 2 and q.shape[1] == self.vectors.shape[1]
        assert r.shape == (q.shape[0], self.m, 2)
        return q, r


def dist(x: np.ndarray, q: np.ndarray) -> float:
    x = np.ascontiguousarray(x)
    q = np.ascontiguousarray(q, dtype=x.dtype)
    f = lib().orc_dist_u8 if x.dtype == np.uint8 else lib().orc_dist_f32
    return float(f(_p(x), _p(q), x.shape[0]))


def pq_table(ix: Index, q) -> np.ndarray:
    """The query's PQ distance table (M x 16 float32)."""
    qq = np.ascontiguousarray(q, dtype=ix.vectors.dtype)
    t = np.zeros(ix.pq_codebook.shape[0] * 16, dtype=np.float32)
    lib().orc_pq_table(C.byref(ix._c), _p(qq), _p(t))
    return t.reshape(-1, 16)


def pq_dist(table: np.ndarray, code: np.ndarray) -> float:
    """Asymmetric distance of one packed code through a query's table."""
    t = np.ascontiguousarray(table, dtype=np.float32)
    c = np.ascontiguousarray(code, dtype=np.uint8)
    return float(lib().orc_pq_dist(_p(t), _p(c), t.shape[0]))


def phi(attr_row, range_row, attr_dtypes) -> int:
    a = np.ascontiguousarray(attr_row, dtype=np.int32)
    r = np.ascontiguousarray(range_row, dtype=np.int32).reshape(-1)
    t = np.ascontiguousarray(attr_dtypes, dtype=np.int32)
    return int(lib().orc_phi(_p(a), _p(r), _p(t), t.shape[0]))


def confident(valid_sq_dists, k: int, eps: float) -> bool:
    v = np.ascontiguousarray(valid_sq_dists, dtype=np.float32)
    if v.size == 0:
        v = np.zeros(1, dtype=np.float32)
        return bool(lib().orc_confident(_p(v), 0, k, eps))
    return bool(lib().orc_confident(_p(v), v.shape[0], k, eps))


def schedule(L0: int, alpha: float, Lmax: int) -> list[int]:
    out = np.zeros(64, dtype=np.int32)
    n = lib().orc_schedule(L0, alpha, Lmax, _p(out), 64)
    assert n > 0
    return [int(x) for x in out[:n]]


@dataclass
class BoaResult:
    ids: np.ndarray        # nq x k uint32
    dists: np.ndarray      # nq x k float32 (squared L2)
    final_L: np.ndarray    # nq int32
    expansions: np.ndarray  # nq int64, summed over phases
    scored: np.ndarray      # nq int64, summed over phases
    phases: list            # per phase: dict(L, active, confident, expansions, scored)


def boa(ix: Index, queries, ranges, k: int, sched: list[int], eps: float = 0.05,
        tau: float = 0.0, threads: int = 1) -> BoaResult:
    """Multi-phase adaptive search of a batch (fixed width: a 1-entry schedule)."""
    q, r = ix._q(queries, ranges)
    nq = q.shape[0]
    s = np.ascontiguousarray(sched, dtype=np.int32)
    ids = np.full((nq, k), PAD, dtype=np.uint32)
    dists = np.full((nq, k), np.inf, dtype=np.float32)
    fl = np.zeros(nq, dtype=np.int32)
    E = np.zeros(nq, dtype=np.int64)
    S = np.zeros(nq, dtype=np.int64)
    st = np.zeros((len(s), 5), dtype=np.int64)
    n = lib().orc_boa(C.byref(ix._c), _p(q), _p(r), nq, k, _p(s), len(s), eps, tau,
                      _p(ids), _p(dists), _p(fl), _p(E), _p(S), _p(st), threads)
    if n < 0:
        raise MemoryError("oracle allocation failed")
    phases = [dict(L=int(a[0]), active=int(a[1]), confident=int(a[2]), expansions=int(a[3]),
                   scored=int(a[4])) for a in st[:n]]
    return BoaResult(ids, dists, fl, E, S, phases)


def boa_warm(ix: Index, queries, ranges, k: int, sched: list[int], eps: float = 0.05) -> BoaResult:
    """Multi-phase search with warm-start escalation (each phase continues
    from the previous phase's list and scored set; see orc_boa_warm)."""
    q, r = ix._q(queries, ranges)
    nq = q.shape[0]
    s = np.ascontiguousarray(sched, dtype=np.int32)
    ids = np.full((nq, k), PAD, dtype=np.uint32)
    dists = np.full((nq, k), np.inf, dtype=np.float32)
    fl = np.zeros(nq, dtype=np.int32)
    E = np.zeros(nq, dtype=np.int64)
    S = np.zeros(nq, dtype=np.int64)
    st = np.zeros((len(s), 5), dtype=np.int64)
    n = lib().orc_boa_warm(C.byref(ix._c), _p(q), _p(r), nq, k, _p(s), len(s), eps,
                           _p(ids), _p(dists), _p(fl), _p(E), _p(S), _p(st))
    if n < 0:
        raise MemoryError("oracle allocation failed")
    phases = [dict(L=int(a[0]), active=int(a[1]), confident=int(a[2]), expansions=int(a[3]),
                   scored=int(a[4])) for a in st[:n]]
    return BoaResult(ids, dists, fl, E, S, phases)


def search_lists(ix: Index, queries, ranges, L: int):
    """Final worklists of a single-width search: (ids, phi, d, len, E, S)."""
    q, r = ix._q(queries, ranges)
    nq = q.shape[0]
    ids = np.zeros((nq, L), dtype=np.uint32)
    ph = np.zeros((nq, L), dtype=np.int32)
    d = np.zeros((nq, L), dtype=np.float32)
    ln = np.zeros(nq, dtype=np.int32)
    E = np.zeros(nq, dtype=np.int64)
    S = np.zeros(nq, dtype=np.int64)
    if lib().orc_search_lists(C.byref(ix._c), _p(q), _p(r), nq, L, _p(ids), _p(ph), _p(d),
                              _p(ln), _p(E), _p(S)) != 0:
        raise MemoryError("oracle allocation failed")
    return ids, ph, d, ln, E, S


def bruteforce(ix: Index, queries, ranges, k: int):
    """Exact filtered top-k: (ids, dists, n_valid)."""
    q, r = ix._q(queries, ranges)
    nq = q.shape[0]
    ids = np.zeros((nq, k), dtype=np.uint32)
    d = np.zeros((nq, k), dtype=np.float32)
    nv = np.zeros(nq, dtype=np.int64)
    lib().orc_bruteforce(C.byref(ix._c), _p(q), _p(r), nq, k, _p(ids), _p(d), _p(nv))
    return ids, d, nv
