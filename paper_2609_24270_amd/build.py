"""Build libasym.so in-tree with hipcc for gfx950 (cross-compiles without a GPU).

    python -m paper_2609_24270_amd.build

Every call recompiles all sources (objects go to paper_2609_24270_amd/_build/).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libasym.so")
ARCH = "gfx950"

SOURCES = ["capi.cpp", "topology.cpp", "topology_cache.cpp", "schedule.cpp", "corun.cpp", "affinity.cpp",
           "interleave.cpp", "kv_place.cpp", "numa_host.cpp",
           "gemm.hip", "gemm_skinny.hip", "attn_decode.hip", "probe.hip", "latency.hip", "copy.hip", "numa.hip",
           "transpose.hip", "noalloc.hip", "mla_decode.hip"]

COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-I", os.path.join(ROOT, "include"), "-Wall", "-Wno-unused-function"]
# Packed fp32 VALU forms are kept out of the device code.
DEVICE_ONLY = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# Per-source extras.  gemm.hip: let the MFMA accumulators take the VGPR form, so
# that the register allocator can keep 256 fp32 accumulators and two sets of
# operand fragments without spilling (the AGPR-only form spills in the k-loop).
# mla_decode.hip: in the AGPR form the 128 output accumulators, which the
# online softmax rescales with vector instructions, were copied between AGPRs
# and VGPRs every 16-token block (256 moves per block); in the VGPR form they
# stay put.  attn_decode.hip: the same, 8 moves per task.
_VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
EXTRA = {"gemm.hip": _VGPR_FORM, "mla_decode.hip": _VGPR_FORM, "attn_decode.hip": _VGPR_FORM}


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found; libasym needs ROCm")
    return p


def _compile(src: str) -> str:
    out = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc()] + COMMON + (DEVICE_ONLY if src.endswith(".hip") else []) + \
        EXTRA.get(src, []) + ["-c", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
