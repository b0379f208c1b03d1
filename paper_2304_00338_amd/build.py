"""Build libmgn.so (gfx950) in-tree with hipcc.

Every HIP source is compiled with ``-Xclang -target-feature -Xclang
-packed-fp32-ops`` (no packed fp32 instructions); the host-only graph code
is compiled without floating-point contraction so the fp64 edge features are
evaluated exactly as documented in include/mgn.h.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmgn.so")
BUILD = os.path.join(ROOT, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

HIP_SOURCES = ["fwd_kernels.hip", "edge_rows.hip", "edge_w160.hip", "node_rows.hip", "node_w160.hip", "enc_rows.hip", "enc_w160.hip", "train_kernels.hip", "bwd_kernels.hip", "misc_kernels.hip", "noalloc.hip", "edge_rows32.hip", "node_rows32.hip"]
HOST_SOURCES = ["graph.cpp", "api.cpp"]

COMMON = ["-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
          "-I", os.path.join(ROOT, "include")]
DEVICE = ["-x", "hip", f"--offload-arch={ARCH}", "-Xclang", "-target-feature",
          "-Xclang", "-packed-fp32-ops"]


def _cmds():
    os.makedirs(BUILD, exist_ok=True)
    cmds, objs = [], []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        cmds.append([HIPCC, *COMMON, *DEVICE, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        extra = ["-ffp-contract=off"] if src == "graph.cpp" else []
        cmds.append([HIPCC, *COMMON, *extra, "-D__HIP_PLATFORM_AMD__", "-c",
                     os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    return cmds, objs


def build(verbose: bool = False) -> str:
    """Compile every source and link libmgn.so; returns its path."""
    cmds, objs = _cmds()
    procs = []
    for c in cmds:
        if verbose:
            print(" ".join(c), flush=True)
        procs.append((c, subprocess.Popen(c, stdout=subprocess.PIPE,
                                          stderr=subprocess.STDOUT, text=True)))
    failed = []
    for c, p in procs:
        out, _ = p.communicate()
        if p.returncode != 0:
            failed.append((c, out))
        elif verbose and out.strip():
            print(out)
    if failed:
        msg = "\n".join(" ".join(c) + "\n" + o for c, o in failed)
        raise RuntimeError("libmgn build failed:\n" + msg)
    link = [HIPCC, "-shared", f"--offload-arch={ARCH}", "-o", LIB + ".tmp", *objs]
    if verbose:
        print(" ".join(link), flush=True)
    r = subprocess.run(link, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("libmgn link failed:\n" + r.stdout)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
