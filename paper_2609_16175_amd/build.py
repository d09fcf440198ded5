"""Build step of libboa.so (hipcc, gfx950). Run by __graft_entry__.build()."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SOURCES = [os.path.join(PKG, "csrc", f) for f in ("boa_kernels.hip", "boa_build.hip", "boa_api.hip")]
LIB = os.path.join(PKG, "libboa.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # distances rely on explicit fused multiply-adds and nothing else fused
    "-ffp-contract=off",
    # no packed-FP32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(PKG, "csrc"),
]


def build(verbose: bool = False, stage_profile: bool = False) -> str:
    """Compile libboa.so; stage_profile=True builds libboa_stageprof.so, a
    variant that prints per-stage cycle counts of every phase to stderr."""
    lib = LIB if not stage_profile else os.path.join(PKG, "libboa_stageprof.so")
    tmp = lib + f".tmp{os.getpid()}"
    cmd = ["hipcc", *HIPCC_FLAGS, *(["-DBOA_STAGE_PROFILE"] if stage_profile else []), *SOURCES, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + r.stdout + r.stderr)
    if verbose:
        print(r.stderr)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
