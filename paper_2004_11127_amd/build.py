"""Build libkred.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

Usage: python -m paper_2004_11127_amd.build   (or call build()).
Objects go to _build/ at the repo root; the library lands next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libkred.so")
PROBE_LIB = os.path.join(PKG, "libkred_probe.so")

SOURCES = ["kred_api.cpp", "k_direct.hip", "k_combine.hip", "k_mfma.hip", "k_mfma64.hip",
           "k_knn.hip", "k_small_mfma.hip", "k_small.hip", "k_cluster.hip"]
PROBE_SOURCES = ["peak_probe.hip"]   # sustained-rate microbenchmarks (bench.py), not the library

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed FP32 VALU instructions stay off: the compiler must not form
# v_pk_{add,mul,fma}_f32 from scalar float code.
FLAGS = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-ffp-contract=fast", "-Wall", "-Wno-unused-function",
         # MFMA results in VGPRs: the epilogues read them at once, and the
         # AGPR form would add a v_accvgpr_read (a VALU slot) per element
         "-mllvm", "-amdgpu-mfma-vgpr-form",
         "-I", INCLUDE, "-I", CSRC]


# sources whose arithmetic must round every operation on its own (the device
# clustering repeats a host construction bit for bit): no fused multiply-adds
NO_CONTRACT = {"k_cluster.hip"}
# sources whose values are never NaN: IEEE mode off, so that fp64 minimum and
# maximum need no quieting of their operands
NO_IEEE = {"k_knn.hip"}


def flags_for(src: str):
    if src in NO_CONTRACT:
        return [f if f != "-ffp-contract=fast" else "-ffp-contract=off" for f in FLAGS]
    if src in NO_IEEE:
        return FLAGS + ["-fno-honor-nans", "-mno-amdgpu-ieee", "-Wno-nan-infinity-disabled"]
    return FLAGS


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC] + flags_for(src) + ["-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    return obj


def _link(objs, lib):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Compile every source and link libkred.so and libkred_probe.so; always rebuilds."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = SOURCES + PROBE_SOURCES
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = dict(zip(srcs, ex.map(_compile, srcs)))
    _link([objs[s] for s in SOURCES], LIB)
    _link([objs[s] for s in PROBE_SOURCES], PROBE_LIB)
    if verbose:
        print("built", LIB, "and", PROBE_LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
