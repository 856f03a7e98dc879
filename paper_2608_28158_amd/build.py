"""In-tree build of libharts.so for gfx950 (hipcc, no JIT cache).

Compiles the host planner and the HIP kernels into
``paper_2608_28158_amd/libharts.so``; the shared object travels with the
source tree, so nothing is built at import time.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(HERE, "libharts.so")
SOURCES = ["plan.cpp", "semantic.cpp", "mbplan.cpp", "kda_plan.cpp", "la.hip", "logp.hip", "conv.hip", "attn.hip",
           "kda.hip"]

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions are generated anywhere in the library
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(verbose: bool = False) -> str:
    """Compile every source and link libharts.so.  Returns its path."""
    objs = []
    obj_dir = os.path.join(HERE, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    for src in SOURCES:
        path = os.path.join(CSRC, src)
        obj = os.path.join(obj_dir, src + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = [hipcc()] + HIP_FLAGS + ["-I", INCLUDE, "-I", CSRC, "-c"] + lang + [path, "-o", obj]
        _run(cmd, verbose)
        objs.append(obj)
    tmp = OUT + ".tmp"
    _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp], verbose)
    os.replace(tmp, OUT)
    return OUT


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout)
        raise RuntimeError(f"build failed: {' '.join(cmd[:3])} ... ({res.returncode})")
    if verbose and res.stdout.strip():
        print(res.stdout)


if __name__ == "__main__":
    print(build(verbose=True))
