"""Compile libswila.so for gfx950 with hipcc (in-tree, no JIT cache).

    python -m paper_2609_39034_amd.build        # or build() from Python
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libswila.so")
# the largest units first, so that the parallel compile ends soonest
SOURCES = ["scan_direct_dk128.hip", "scan_direct_dk64.hip", "scan_pipe.hip",
           "scan_pipe_temporal.hip", "scan_direct_dk32.hip", "scan_direct_dk16.hip",
           "scan_pipe_newton.hip", "scan_gated_chunk.hip", "decode.hip", "scan_backward.hip",
           "scan_direct.hip", "swila_api.hip"]
ARCH = "gfx950"

# Packed fp32 VALU instructions are turned off for every kernel: the compiler
# still emits ordinary fp32 FMAs.
CFLAGS = ["-std=c++17", "-O3", "--offload-arch=" + ARCH, "-fPIC", "-Wall",
          "-Wno-unused-result", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I" + INCLUDE, "-I" + CSRC]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


# Per-file additions.  The chunk scan never relies on NaN semantics (inputs
# are finite; idle lanes' values are never stored), which lets the compiler
# fold the cross-lane DPP moves into v_max/v_add.
EXTRA = {f: ["-fno-honor-nans"] for f in ("scan_pipe.hip", "scan_pipe_newton.hip",
                                          "scan_pipe_temporal.hip")}


def _compile(src, verbose):
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc()] + CFLAGS + EXTRA.get(src, []) + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s%s" % (src, r.stdout, r.stderr))
    return obj


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every HIP source and link libswila.so; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 1)
    with concurrent.futures.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s%s" % (r.stdout, r.stderr))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
