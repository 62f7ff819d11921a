"""Build libnmt.so (HIP, gfx950 only) in-tree with hipcc.

Usage: ``python -m paper_1605_04809_amd.build``.  Every call recompiles.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libnmt.so")
SOURCES = ("kernels.hip", "api.hip", "forest.hip")
HOST_SOURCES = ("forest_host.cpp",)   # plain C++, compiled by the host compiler

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX", "g++")
# Packed-FP32 VALU instructions are disabled for all device code.
FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-munsafe-fp-atomics"]


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile libnmt.so; ``defines`` (e.g. ``["NMT_GRU_TM=64"]``) override tile constants."""
    if not os.path.exists(HIPCC) and shutil.which("hipcc") is None:
        raise RuntimeError("hipcc not found; libnmt needs ROCm to build")
    hipcc = HIPCC if os.path.exists(HIPCC) else shutil.which("hipcc")
    tmp = tempfile.mkdtemp(prefix="nmt_build_")
    try:
        objs = []
        for src in SOURCES:
            obj = os.path.join(tmp, src.replace(".hip", ".o"))
            cmd = [hipcc, *FLAGS, *[f"-D{d}" for d in defines], "-c", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr[-6000:]}")
            objs.append(obj)
        for src in HOST_SOURCES:
            obj = os.path.join(tmp, src.replace(".cpp", ".o"))
            cmd = [CXX, "-O2", "-std=c++17", "-fPIC", "-Wall", "-I", "/opt/rocm/include", "-c",
                   os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"{CXX} failed on {src}:\n{r.stderr[-6000:]}")
            objs.append(obj)
        out_tmp = out + ".tmp"
        cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", out_tmp]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{r.stderr[-4000:]}")
        os.replace(out_tmp, out)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
