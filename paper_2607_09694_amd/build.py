"""Build of the gfx950 routing library (hipcc, in-tree shared object)."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "liblrattnres.so")
SOURCES = ["route_fwd.hip", "route_bwd.hip", "route_block.hip", "route_all.hip",
           "route_all_bwd.hip", "key_proj.hip", "key_proj_bwd.hip", "route_plan.cpp", "capi.cpp"]
# Benchmark-only helper: streaming copy / read kernels of known traffic.
PROBE_LIB = os.path.join(PKG, "libhbmprobe.so")
PROBE_SOURCES = ["hbm_probe.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# gfx950 only.  Packed fp32 VALU ops are disabled for every HIP translation
# unit (the compiler would otherwise form v_pk_{add,mul,fma}_f32 by itself).
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE, "-I", CSRC]


def build(verbose: bool = False) -> str:
    """Compile every source and link liblrattnres.so (and the benchmark's
    libhbmprobe.so) next to this file."""
    _build_lib(SOURCES, LIB, verbose)
    _build_lib(PROBE_SOURCES, PROBE_LIB, verbose)
    return LIB


def _build_lib(sources, lib, verbose):
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{res.stderr}")
        if verbose and res.stderr.strip():
            print(res.stderr, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max_workers=len(sources)) as ex:
        objs = list(ex.map(compile_one, sources))
    tmp = lib + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, lib)


if __name__ == "__main__":
    print(build(verbose=True))
