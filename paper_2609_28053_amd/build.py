"""Build libeqb.so for gfx950 with hipcc, in place next to this file.

    python -m paper_2609_28053_amd.build          # or: python paper_2609_28053_amd/build.py
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = [os.path.join(CSRC, f) for f in ("eqb_api.hip", "margin.hip", "select.hip", "balance.hip", "variants.hip",
                                          "layer_noalloc.hip")]
# The routing kernels are compiled on their own, without IEEE mode: their
# float maxima and medians then need no NaN quieting, which lets the compiler
# fold each DPP group maximum into one instruction and schedule around its
# wait states.  Their operands are keys and finite scores, never NaN (finite
# inputs are a precondition of the library).
ROUTE_SOURCE = os.path.join(CSRC, "route.hip")
ROUTE_FLAGS = ["-mno-amdgpu-ieee", "-fno-honor-nans"]
OUT = os.path.join(HERE, "libeqb.so")
ARCH = os.environ.get("EQB_OFFLOAD_ARCH", "gfx950")

FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-ffp-contract=off",               # no fused multiply-add anywhere on the path
    # packed FP32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    if verbose and res.stderr:
        sys.stderr.write(res.stderr)


def build(verbose: bool = False, extra=()) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = OUT + ".tmp"
    route_obj = OUT + ".route.o"
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    compile_flags = [f for f in FLAGS if f != "-shared"]
    try:
        _run([hipcc, *compile_flags, *ROUTE_FLAGS, *extra, *inc, "-c", ROUTE_SOURCE, "-o", route_obj], verbose)
        _run([hipcc, *FLAGS, *extra, *inc, *SOURCES, "-x", "none", route_obj, "-o", tmp], verbose)
    finally:
        if os.path.exists(route_obj):
            os.remove(route_obj)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True, extra=sys.argv[1:]))
