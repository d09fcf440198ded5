"""MI355X-native BOA: batched filtered beam search with online beamwidth
adaptation ("BOA: Beamwidth Online Adaptation for Filtered-ANNS on a GPU").

Thin ctypes binding of libboa.so (include/boa.h): argument marshalling
only. Every step of the search runs in the library's HIP kernels; torch
provides device memory and the stream. The library is loaded on first
use; where libboa.so is not built, that first use raises ImportError:
there is no CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# BOA_LIB selects another build of the same library (e.g. the stage-profiling
# variant libboa_stageprof.so); default: the product build.
LIB_PATH = os.path.join(_HERE, os.environ.get("BOA_LIB", "libboa.so"))

VEC_F32, VEC_U8 = 0, 1
ATTR_I32, ATTR_F32 = 0, 1
PAD = 0xFFFFFFFF
MAX_PHASES = 32
ERRORS = {0: "BOA_OK", -1: "BOA_EINVAL", -2: "BOA_ENOMEM", -3: "BOA_EHIP", -4: "BOA_EUNSUPPORTED",
          -5: "BOA_EOVERFLOW"}


class BoaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class Params(C.Structure):
    _fields_ = [("k", C.c_int32), ("L0", C.c_int32), ("Lmax", C.c_int32), ("alpha", C.c_double),
                ("eps", C.c_double), ("tau", C.c_double), ("fixed_L", C.c_int32),
                ("boa_plus", C.c_int32), ("sub_batches", C.c_int32), ("lds_hash_slots", C.c_int32),
                ("schedule", C.POINTER(C.c_int32)), ("n_schedule", C.c_int32), ("fused", C.c_int32),
                ("warm_start", C.c_int32), ("pq", C.c_int32), ("escalation_waves", C.c_int32)]


class BuildParams(C.Structure):
    _fields_ = [("alpha", C.c_double), ("attr_levels", C.c_int32)]


class PhaseStats(C.Structure):
    _fields_ = [("L", C.c_int32), ("active", C.c_int32), ("confident", C.c_int32),
                ("launches", C.c_int32), ("expansions", C.c_int64), ("scored", C.c_int64),
                ("gathered_bytes", C.c_double), ("kernel_ms", C.c_float)]


class Stats(C.Structure):
    _fields_ = [("n_phases", C.c_int32), ("waves_per_block", C.c_int32), ("blocks", C.c_int32),
                ("lds_hash_slots", C.c_int32), ("spilled_queries", C.c_int64), ("total_ms", C.c_float),
                ("cum_searches", C.c_int64), ("cum_launches", C.c_int64), ("cum_kernel_ms", C.c_double),
                ("phase", PhaseStats * MAX_PHASES),
                ("cum_phase_launches", C.c_int64 * MAX_PHASES), ("cum_phase_kernel_ms", C.c_double * MAX_PHASES)]


_lib = None


def lib():
    """The loaded libboa.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                              "(hipcc --offload-arch=gfx950). There is no CPU fallback.")
        L = C.CDLL(LIB_PATH)
        P = C.c_void_p
        L.boa_build_index_from_arrays.restype = C.c_int
        L.boa_build_index_from_arrays.argtypes = [P, C.c_int64, C.c_int32, C.c_int32, P, C.c_int32, P,
                                                  P, C.c_int32, C.c_int64, C.POINTER(P)]
        L.boa_search.restype = C.c_int
        L.boa_search.argtypes = [P, P, P, C.c_int64, C.POINTER(Params), P, P, P, P, P, P]
        L.boa_search_noalloc.restype = C.c_int
        L.boa_search_noalloc.argtypes = [P, P, P, C.c_int64, C.POINTER(Params), P, P, P, P, P, P]
        L.boa_get_stats.restype = C.c_int
        L.boa_get_stats.argtypes = [P, C.POINTER(Stats)]
        L.boa_reset_counters.restype = C.c_int
        L.boa_reset_counters.argtypes = [P]
        L.boa_build_index_ex.restype = C.c_int
        L.boa_build_index_ex.argtypes = [P, C.c_int64, C.c_int32, C.c_int32, P, C.c_int32, P,
                                         P, C.c_int32, C.c_int64, C.POINTER(BuildParams), C.POINTER(P)]
        L.boa_default_build_params.restype = None
        L.boa_default_build_params.argtypes = [C.POINTER(BuildParams)]
        L.boa_set_pq.restype = C.c_int
        L.boa_set_pq.argtypes = [P, P, P, C.c_int32]
        L.boa_get_graph.restype = C.c_int
        L.boa_get_graph.argtypes = [P, P, C.POINTER(C.c_int64), C.POINTER(C.c_int64)]
        L.boa_free_index.restype = None
        L.boa_free_index.argtypes = [P]
        L.boa_last_error.restype = C.c_char_p
        L.boa_last_error.argtypes = []
        L.boa_default_params.restype = None
        L.boa_default_params.argtypes = [C.POINTER(Params)]
        _lib = L
    return _lib


def _check(rc: int):
    if rc != 0:
        raise BoaError(rc, lib().boa_last_error().decode())


def default_params() -> Params:
    p = Params()
    lib().boa_default_params(C.byref(p))
    return p


@dataclass
class SearchResult:
    ids: "object"        # torch int32 (nq, k); -1 (0xFFFFFFFF) marks padding
    dists: "object"      # torch float32 (nq, k) squared L2
    final_L: "object"    # torch int32 (nq,)
    expansions: "object" = None
    scored: "object" = None


class Index:
    """A graph index resident in device memory (owned by libboa)."""

    def __init__(self, vectors: np.ndarray, attrs: np.ndarray, attr_dtypes, adjacency, entry: int = -1,
                 R: int = 0, alpha: float = 1.2, attr_levels: int = 4):
        """adjacency: n x R uint32 rows, or None to have the library build the
        graph with R edges per row (alpha, attr_levels: boa_build_params);
        entry: the entry point, or -1 for the medoid (computed by the library)."""
        vectors = np.ascontiguousarray(vectors)
        if vectors.dtype == np.float32:
            vt = VEC_F32
        elif vectors.dtype == np.uint8:
            vt = VEC_U8
        else:
            raise TypeError("vectors must be float32 or uint8")
        attrs = np.ascontiguousarray(attrs, dtype=np.int32)
        types = np.ascontiguousarray(attr_dtypes, dtype=np.int32)
        n, d = vectors.shape
        if adjacency is None:
            adj, width, aptr = None, int(R), None
        else:
            adj = np.ascontiguousarray(adjacency, dtype=np.uint32)
            width, aptr = adj.shape[1], adj.ctypes.data
            if adj.shape[0] != n:
                raise ValueError("shape mismatch between vectors and adjacency")
        if attrs.shape != (n, types.shape[0]):
            raise ValueError("shape mismatch between vectors and attributes")
        h = C.c_void_p()
        bp = BuildParams()
        lib().boa_default_build_params(C.byref(bp))
        bp.alpha, bp.attr_levels = alpha, attr_levels
        _check(lib().boa_build_index_ex(vectors.ctypes.data, n, d, vt, attrs.ctypes.data,
                                        types.shape[0], types.ctypes.data, aptr,
                                        width, int(entry), C.byref(bp), C.byref(h)))
        self._h = h
        self.n, self.d, self.m, self.R = n, d, types.shape[0], width
        self.vec_dtype = vt

    def set_pq(self, codebook: np.ndarray, codes: np.ndarray):
        """Product-quantisation data: codebook M x 16 x d/M float32, codes
        n x M/2 uint8 (workloads.pq layout)."""
        cb = np.ascontiguousarray(codebook, dtype=np.float32)
        cc = np.ascontiguousarray(codes, dtype=np.uint8)
        M = cb.shape[0]
        if cb.shape != (M, 16, self.d // M) or cc.shape != (self.n, M // 2):
            raise ValueError("codebook must be M x 16 x d/M and codes n x M/2")
        _check(lib().boa_set_pq(self._h, cb.ctypes.data, cc.ctypes.data, M))

    def graph(self):
        """(adjacency n x R uint32, entry, repaired): the graph the index
        searches; repaired counts the in-edges the library's construction
        added to reach every point (-1 when the caller gave the graph)."""
        adj = np.empty((self.n, self.R), dtype=np.uint32)
        e, rep = C.c_int64(), C.c_int64()
        _check(lib().boa_get_graph(self._h, adj.ctypes.data, C.byref(e), C.byref(rep)))
        return adj, int(e.value), int(rep.value)

    def close(self):
        if getattr(self, "_h", None):
            lib().boa_free_index(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def search(self, queries, ranges, k: int, L0: int = 16, Lmax: int = 512, alpha: float = 2.0,
               eps: float = 0.05, tau: float = 0.0, fixed_L: int = 0, boa_plus: bool = False,
               sub_batches: int = 10, lds_hash_slots: int = 0, schedule=None, fused: bool = False,
               split: bool = False, counters: bool = False,
               stream=None, out=None, no_alloc: bool = False, warm: bool = False,
               pq: bool = False, escalation_waves: int = 0) -> SearchResult:
        """Adaptive filtered top-k of a batch of device-resident queries.

        queries: torch tensor (nq, d) on the GPU, float32 or uint8 like the index.
        ranges:  torch int32 tensor (nq, m, 2) on the GPU (float32 columns as bit patterns).
        fused:   every phase in one persistent launch; split: the first phase in
                 one launch, the survivors through all later phases in a second.
        warm:    warm-start escalation (fused mode): each phase continues from
                 the previous phase's list and visited set.
        pq:      traverse with product-quantised distances (set_pq first) and
                 re-rank each phase's valid entries exactly.
        escalation_waves: split mode: 0 two waves per query in the escalation
                 launch where it applies, 1 one wave per query.
        no_alloc: call boa_search_noalloc (the library allocates no device
                 memory for the call; pass preallocated `out` tensors to
                 allocate nothing on the torch side either).
        """
        import torch
        if not (queries.is_cuda and ranges.is_cuda):
            raise ValueError("queries and ranges must be device tensors")
        want = torch.float32 if self.vec_dtype == VEC_F32 else torch.uint8
        if queries.dtype != want or queries.dim() != 2 or queries.shape[1] != self.d:
            raise ValueError(f"queries must be ({'{'}nq{'}'}, {self.d}) {want}")
        if ranges.dtype != torch.int32 or tuple(ranges.shape) != (queries.shape[0], self.m, 2):
            raise ValueError(f"ranges must be int32 of shape (nq, {self.m}, 2)")
        queries = queries.contiguous()
        ranges = ranges.contiguous()
        nq = queries.shape[0]
        dev = queries.device
        if out is None:
            ids = torch.empty((nq, k), dtype=torch.int32, device=dev)
            dists = torch.empty((nq, k), dtype=torch.float32, device=dev)
            fl = torch.empty((nq,), dtype=torch.int32, device=dev)
            E = torch.empty((nq,), dtype=torch.int32, device=dev) if counters else None
            S = torch.empty((nq,), dtype=torch.int32, device=dev) if counters else None
        else:
            ids, dists, fl, E, S = out
        p = default_params()
        p.k, p.L0, p.Lmax, p.alpha, p.eps, p.tau = k, L0, Lmax, alpha, eps, tau
        p.fixed_L, p.boa_plus, p.sub_batches, p.lds_hash_slots = fixed_L, int(boa_plus), sub_batches, lds_hash_slots
        if fused and split:
            raise ValueError("fused and split are exclusive")
        p.fused = 2 if split else int(fused)
        p.warm_start = int(warm)
        p.pq = int(pq)
        p.escalation_waves = int(escalation_waves)
        sched_arr = None
        if schedule is not None:
            sched_arr = (C.c_int32 * len(schedule))(*schedule)
            p.schedule = C.cast(sched_arr, C.POINTER(C.c_int32))
            p.n_schedule = len(schedule)
        st = (stream if stream is not None else torch.cuda.current_stream(dev)).cuda_stream
        fn = lib().boa_search_noalloc if no_alloc else lib().boa_search
        _check(fn(self._h, queries.data_ptr(), ranges.data_ptr(), nq, C.byref(p),
                                ids.data_ptr(), dists.data_ptr(), fl.data_ptr(),
                                E.data_ptr() if E is not None else None,
                                S.data_ptr() if S is not None else None, st))
        return SearchResult(ids, dists, fl, E, S)

    def stats(self) -> dict:
        s = Stats()
        _check(lib().boa_get_stats(self._h, C.byref(s)))
        phases = []
        for i in range(s.n_phases):
            ph = s.phase[i]
            phases.append(dict(L=ph.L, active=ph.active, confident=ph.confident, launches=ph.launches,
                               expansions=ph.expansions, scored=ph.scored,
                               gathered_bytes=ph.gathered_bytes, kernel_ms=ph.kernel_ms))
        return dict(phases=phases, waves_per_block=s.waves_per_block, blocks=s.blocks,
                    lds_hash_slots=s.lds_hash_slots, spilled_queries=s.spilled_queries,
                    total_ms=s.total_ms, cum_searches=s.cum_searches, cum_launches=s.cum_launches,
                    cum_kernel_ms=s.cum_kernel_ms,
                    cum_phase_launches=[int(s.cum_phase_launches[i]) for i in range(s.n_phases)],
                    cum_phase_kernel_ms=[float(s.cum_phase_kernel_ms[i]) for i in range(s.n_phases)])

    def reset_counters(self):
        _check(lib().boa_reset_counters(self._h))
