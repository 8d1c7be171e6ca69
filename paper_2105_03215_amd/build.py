"""Builds libbyoc.so (the C-ABI library) in-tree with hipcc for gfx950.

Usage: python -m paper_2105_03215_amd.build   (or call build()).
"""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libbyoc.so")
ROOT = os.path.dirname(PKG)

SOURCES = ["json.cpp", "graph.cpp", "capi.cpp", "engine.cpp", "conv_mfma.hip", "conv_dma.hip", "conv_halo.hip", "bottleneck.hip", "ir_block.hip", "stem.hip", "dense_rows.hip", "conv_f32.hip",
           "vector_ops.hip", "conv_i8.hip", "quant.hip", "static_scratch.hip"]

# -packed-fp32-ops: keep the compiler from emitting packed fp32 ALU ops.
FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall",
         "-Wno-unused-result", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + os.path.join(ROOT, "include")]


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src, hipcc, verbose):
    out = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc] + FLAGS + ["-c", os.path.join(CSRC, src), "-o", out]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines()
            if "packed-fp32-ops' is not a recognized feature" not in ln]
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s" % (src, "\n".join(msgs)))
    if verbose and msgs:
        print("\n".join(msgs))
    return out


def build(verbose=False, jobs=None):
    """Compile every source and link libbyoc.so; always rebuilds."""
    hipcc = _hipcc()
    os.makedirs(OBJ, exist_ok=True)
    jobs = jobs or min(8, os.cpu_count() or 4)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, hipcc, verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
