"""Build libfp8lin.so (HIP, gfx950) in-tree with hipcc.

Usage: python -m paper_2309_17224_amd.build   (or call build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libfp8lin.so")
SOURCES = ["fp8lin_api.hip", "fp8lin_amax_cast.hip", "fp8lin_gemm.hip", "fp8lin_decoder.hip"]
# measurement aid beside the library (bench.py --mfma-ceiling), not the method
PROBE_LIB = os.path.join(PKG, "libfp8probe.so")
PROBE_SOURCE = "fp8probe.hip"
ARCH = "gfx950"


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def flags() -> list[str]:
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
        # no packed-fp32 instructions in device code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", INCLUDE, "-I", CSRC,
    ]


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every source (in parallel) and link libfp8lin.so next to this file."""
    from concurrent.futures import ThreadPoolExecutor
    obj_dir = os.path.join(PKG, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    objs = [os.path.join(obj_dir, src.replace(".hip", ".o")) for src in SOURCES]
    cmds = [[hipcc()] + flags() + ["-c", os.path.join(CSRC, src), "-o", obj] for src, obj in zip(SOURCES, objs)]
    probe_tmp = PROBE_LIB + ".tmp%d" % os.getpid()
    cmds.append([hipcc()] + flags() + ["-shared", os.path.join(CSRC, PROBE_SOURCE), "-o", probe_tmp])
    if verbose:
        for cmd in cmds:
            print(" ".join(cmd), flush=True)
    jobs = jobs or min(len(cmds), max(1, (os.cpu_count() or 1) // 2))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        for r in ex.map(lambda c: subprocess.run(c, check=True), cmds):
            pass
    os.replace(probe_tmp, PROBE_LIB)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
