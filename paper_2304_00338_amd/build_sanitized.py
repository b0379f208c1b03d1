"""Host-sanitizer build of libmgn for CPU testing.

The host-side C++ (graph construction, partition, patch extraction and
union, tile schedule, context planning in api.cpp, the no-alloc entry's
host checks) is compiled with AddressSanitizer and UndefinedBehaviorSanitizer
on the host side only; the device objects of the normal build are linked in
unchanged (no GPU code is sanitized).  The library is written to
_build/sanitized/libmgn.so; run_host_tests() runs the CPU host-library tests
against it in a child process with the ASan runtime preloaded.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

from . import build as B

OUT = os.path.join(B.BUILD, "sanitized")
LIB = os.path.join(OUT, "libmgn.so")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def asan_runtime() -> str:
    r = subprocess.run([B.HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], stdout=subprocess.PIPE,
                       stderr=subprocess.DEVNULL, text=True)
    p = r.stdout.strip()
    if not os.path.isabs(p) or not os.path.exists(p):
        cands = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
        if not cands:
            raise RuntimeError("ASan runtime not found")
        p = cands[0]
    return p


def build() -> str:
    """Compile the host sources with the sanitizers and link them with the
    device objects of the normal build (built first if missing)."""
    os.makedirs(OUT, exist_ok=True)
    _, objs = B._cmds()
    if not all(os.path.exists(o) for o in objs):
        B.build()
    hip_objs = [o for o in objs if o.endswith(".hip.o")]
    host = []
    for src in B.HOST_SOURCES:
        obj = os.path.join(OUT, src + ".o")
        extra = ["-ffp-contract=off"] if src == "graph.cpp" else []
        cmd = [B.HIPCC, *B.COMMON, *extra, *SAN, "-D__HIP_PLATFORM_AMD__", "-c", os.path.join(B.CSRC, src),
               "-o", obj]
        subprocess.run(cmd, check=True)
        host.append(obj)
    link = [B.HIPCC, "-shared", f"--offload-arch={B.ARCH}", "-fsanitize=address", "-fsanitize=undefined",
            "-fno-gpu-sanitize", "-shared-libsan", "-o", LIB, *hip_objs, *host]
    subprocess.run(link, check=True)
    return LIB


def run_host_tests(tests=("tests/test_host_lib.py",)) -> int:
    """Run the CPU host-library tests against the sanitized library (the ASan
    runtime preloaded into a child Python); returns its exit status."""
    env = dict(os.environ)
    env["MGN_LIB"] = LIB
    env["LD_PRELOAD"] = asan_runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:verify_asan_link_order=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu", *tests]
    return subprocess.run(cmd, cwd=B.ROOT, env=env).returncode


if __name__ == "__main__":
    print(build())
    sys.exit(run_host_tests())
