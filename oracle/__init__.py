"""CPU oracle for the hot path.  TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never imports, links or calls it,
and it imports nothing from the product package: the two sides share only the
seeded input generators, which hold none of the method's arithmetic.

Contents
  gemm_bf16          plain C GEMM, fp32 k-ordered accumulation, bf16 RNE output
                     (the full-GPU kernel case of Section 7.1 computes this
                     product; placement changes only who computes each tile)
  grouped_gemm_bf16  one gemm_bf16 per group of packed rows (the grouped GEMM
                     of Section 7.1, the mixture-of-experts expert layer)
  f32_to_bf16        the oracle's own round-to-nearest-even conversion
  schedule           per-partition work quotas proportional to compute units
                     (Section 7.1 and the full-GPU lesson of Section 7.4)
  topology           the topology map's definition and exact invariants
                     (Section 5.1 topology discovery, Appendix G affinity)
  affinity           XCD groups and home groups from per-address latencies
                     (Section 6.1, Appendix G)
  interleave         partition-hash bits from one- and two-bit address flips
                     (Section 6.1, NUMA partition identification)
  numa               chunk homes of an allocation and the local / remote read
                     lists (Section 6.1 local and remote bandwidth)
  attention          decode attention with grouped key/value heads, one
                     float64 softmax per (request, head) (Section 7.1)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle_gemm.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

# Plain -O2 build: no -ffast-math, no contraction, OpenMP over output rows.
BUILD_CMD = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
             "-fPIC", "-shared", "-std=c11", _SRC, "-o", _LIB_PATH]


def build() -> str:
    """Compile liboracle.so with gcc (always recompiles)."""
    tmp = _LIB_PATH + ".tmp"
    cmd = BUILD_CMD[:-1] + [tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    u16p = ctypes.POINTER(ctypes.c_uint16)
    f32p = ctypes.POINTER(ctypes.c_float)
    lib.oracle_gemm_bf16.argtypes = [
        ctypes.c_int, ctypes.c_int, ctypes.c_int, u16p, ctypes.c_int, u16p,
        ctypes.c_int, ctypes.c_int, f32p, u16p]
    lib.oracle_gemm_bf16.restype = ctypes.c_int
    lib.oracle_f32_to_bf16_array.argtypes = [f32p, u16p, ctypes.c_int64]
    lib.oracle_f32_to_bf16_array.restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _u16(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint16))


def gemm_bf16(A_bits: np.ndarray, B_bits: np.ndarray, b_layout: str = "nk",
              want_r32: bool = True):
    """C = A . B with fp32 k-ordered accumulation and bf16 RNE output.

    A_bits: uint16 [M, K] bf16 bit patterns (row-major).
    B_bits: uint16 [N, K] for b_layout "nk" (B stored transposed, K-contiguous)
            or [K, N] for "kn".
    Returns (R32 float32 [M, N] or None, C uint16 [M, N] bf16 bits).
    """
    A = np.ascontiguousarray(A_bits, dtype=np.uint16)
    B = np.ascontiguousarray(B_bits, dtype=np.uint16)
    M, K = A.shape
    if b_layout == "nk":
        N, K2 = B.shape
        lay, ldb = 0, K
    elif b_layout == "kn":
        K2, N = B.shape
        lay, ldb = 1, N
    else:
        raise ValueError("b_layout must be 'nk' or 'kn'")
    if K2 != K:
        raise ValueError(f"inner dimensions differ: A has K={K}, B has K={K2}")
    R = np.empty((M, N), dtype=np.float32) if want_r32 else None
    C = np.empty((M, N), dtype=np.uint16)
    lib = _load()
    rc = lib.oracle_gemm_bf16(
        M, N, K, _u16(A), max(K, 1), _u16(B), max(ldb, 1), lay,
        R.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if R is not None else None,
        _u16(C))
    if rc != 0:
        raise RuntimeError("oracle_gemm_bf16 failed")
    return R, C


def grouped_gemm_bf16(A_bits: np.ndarray, B_bits: np.ndarray, M, want_r32: bool = True):
    """Grouped GEMM, by definition one gemm_bf16 per group.

    A_bits: uint16 [sum(M), K], the groups' rows packed in group order.
    B_bits: uint16 [G, N, K], group g's weights stored [N, K].
    M:      the G row counts (>= 0).
    Returns (R32 float32 [sum(M), N] or None, C uint16 [sum(M), N]), packed
    like A: group g's rows start at M[0] + ... + M[g-1].
    """
    A = np.asarray(A_bits, dtype=np.uint16)
    B = np.asarray(B_bits, dtype=np.uint16)
    G, N, K = B.shape
    if len(M) != G or A.shape != (sum(M), K):
        raise ValueError("A must be [sum(M), K] and B [len(M), N, K]")
    R = np.zeros((A.shape[0], N), dtype=np.float32) if want_r32 else None
    C = np.zeros((A.shape[0], N), dtype=np.uint16)
    row = 0
    for g, m in enumerate(M):
        if m:
            Rg, Cg = gemm_bf16(A[row:row + m], B[g], "nk", want_r32)
            C[row:row + m] = Cg
            if want_r32:
                R[row:row + m] = Rg
        row += m
    return R, C


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """The oracle's fp32 -> bf16 round-to-nearest-even, returned as uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty(x.shape, dtype=np.uint16)
    _load().oracle_f32_to_bf16_array(
        x.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), _u16(y), x.size)
    return y


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def num_threads() -> int:
    return int(_load().oracle_num_threads())
