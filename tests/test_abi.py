"""The C-ABI library loads and exports what include/boa.h declares; host-side
validation returns error codes without touching a device."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_2609_16175_amd as boa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "boa.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(boa_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("boa_build_index_from_arrays", "boa_search", "boa_get_stats", "boa_free_index",
                 "boa_last_error", "boa_default_params"):
        assert want in names


def test_library_exports_every_declared_symbol():
    lib = C.CDLL(boa.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_struct_layouts_match_header():
    # sizes follow from the header's field order on x86-64
    # k, L0, Lmax, pad, alpha, eps, tau, fixed_L, boa_plus, sub_batches,
    # lds_hash_slots, schedule, n_schedule, fused, warm_start, pq,
    # escalation_waves, tail padding to the struct's 8-byte alignment
    assert C.sizeof(boa.Params) == 4 * 3 + 4 + 8 * 3 + 4 * 4 + 8 + 4 + 4 + 4 + 4 + 4 + 4
    assert boa.Params.warm_start.offset == 72 and boa.Params.pq.offset == 76
    assert boa.Params.escalation_waves.offset == 80
    assert C.sizeof(boa.PhaseStats) == 4 * 4 + 8 * 2 + 8 + 4 + 4


def test_default_params():
    p = boa.default_params()
    assert (p.k, p.L0, p.Lmax, p.alpha, p.eps, p.tau) == (10, 16, 512, 2.0, 0.05, 0.0)
    assert p.fixed_L == 0 and p.boa_plus == 0 and p.sub_batches == 10
    assert p.escalation_waves == 0


def _build(**over):
    n, d, m, R = 50, 8, 2, 4
    args = dict(vectors=np.zeros((n, d), np.float32), n=n, d=d, vt=boa.VEC_F32,
                attrs=np.zeros((n, m), np.int32), m=m, types=np.zeros(m, np.int32),
                adj=np.full((n, R), boa.PAD, np.uint32), R=R, entry=0)
    args.update(over)
    h = C.c_void_p()
    ptr = lambda a: a.ctypes.data if isinstance(a, np.ndarray) else a
    rc = boa.lib().boa_build_index_from_arrays(ptr(args["vectors"]), args["n"], args["d"], args["vt"],
                                               ptr(args["attrs"]), args["m"], ptr(args["types"]),
                                               ptr(args["adj"]), args["R"], args["entry"], C.byref(h))
    return rc, boa.lib().boa_last_error().decode()


@pytest.mark.parametrize("over,needle", [
    (dict(vectors=None), "NULL"),
    (dict(n=0), "n out of range"),
    (dict(n=1 << 24), "n out of range"),
    (dict(d=6), "d % 4"),
    (dict(d=2048), "d out of range"),
    (dict(vt=7), "vec_dtype"),
    (dict(m=9), "m out of range"),
    (dict(R=65), "R out of range"),
    (dict(entry=50), "entry"),
    (dict(types=np.array([0, 5], np.int32)), "dtype"),
    (dict(adj=np.full((50, 4), 50, np.uint32)), "adjacency id out of range"),
    (dict(adj=np.tile(np.arange(50, dtype=np.uint32)[:, None], (1, 4))), "its own id"),
    (dict(adj=np.tile(np.array([[30, 9, 30, 0xFFFFFFFF]], dtype=np.uint32), (50, 1))), "twice"),
])
def test_build_validation(over, needle):
    rc, msg = _build(**over)
    assert rc == -1 and needle in msg


def test_build_without_adjacency_beyond_the_build_limit_is_unsupported():
    # the library builds the graph itself only up to BOA_MAX_BUILD_N points;
    # refused before any array is read or any device work
    rc, msg = _build(adj=None, n=(2 << 20) + 1)
    assert rc == -4 and "BOA_MAX_BUILD_N" in msg


def test_entry_below_minus_one_is_invalid():
    rc, msg = _build(entry=-2)
    assert rc == -1 and "entry" in msg


def test_search_null_index():
    p = boa.default_params()
    rc = boa.lib().boa_search(None, None, None, 0, C.byref(p), None, None, None, None, None, None)
    assert rc == -1


def test_missing_library_fails_loudly():
    # no fallback: with the library absent, the binding refuses to run
    import subprocess
    import sys
    code = ("import paper_2609_16175_amd as boa\n"
            "try:\n    boa.lib()\nexcept ImportError as e:\n    print('refused:', e)\n"
            "else:\n    print('loaded')\n")
    env = dict(os.environ, BOA_LIB="libboa_missing_for_test.so")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                       cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))), timeout=120)
    assert "refused:" in r.stdout and "is not built" in r.stdout, r.stdout + r.stderr
