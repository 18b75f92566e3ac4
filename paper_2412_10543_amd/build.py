"""Builds librag_attn.so (gfx950) in-tree with hipcc.

    python -m paper_2412_10543_amd.build        # or __graft_entry__.build()
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "librag_attn.so")
OBJDIR = os.path.join(PKG, "_build")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed fp32 VALU instructions are kept out of every kernel.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
          "-Wall", "-Wno-unused-result"]

# Per-source device flags.  The int4 GEMM keeps its MFMA accumulators in
# ordinary VGPRs, where the per-group rescaling (a VALU multiply) can reach
# them without AGPR copies.
SOURCE_FLAGS = {"awq_gemm.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}
SOURCES = ["kernels.hip", "kv_cache.hip", "awq_gemm.hip", "decode_scratch.hip", "api.cpp",
           "awq_api.cpp", "planner.cpp"]
HEADERS = ["common.h", "prefill_tile.h", "decode_unit.h", "launch.h", "errors.h", "awq.h"]


PROBES = os.path.join(PKG, "libceiling_probes.so")


def build_probes(verbose: bool = False) -> str:
    """The hardware ceiling probes (measurement only, not the method)."""
    os.makedirs(OBJDIR, exist_ok=True)
    obj = os.path.join(OBJDIR, "ceiling_probes.o")
    cmd = [HIPCC, *COMMON, *DEVICE_FLAGS, "-x", "hip", "-c",
           os.path.join(CSRC, "ceiling_probes.hip"), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True, stderr=None if verbose else subprocess.PIPE)
    tmp = PROBES + ".tmp"
    subprocess.run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, obj], check=True)
    os.replace(tmp, PROBES)
    return PROBES


def build(verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else ["-x", "hip"]
        cmd = [HIPCC, *COMMON, *DEVICE_FLAGS, *SOURCE_FLAGS.get(src, []), *lang, "-c",
               os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True, stderr=None if verbose else subprocess.PIPE)
        objs.append(obj)
    tmp = LIBRARY + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIBRARY)
    build_probes(verbose)
    return LIBRARY


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIBRARY)
