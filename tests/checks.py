"""Shared test-side comparison helpers (no method arithmetic).

The GEMM gate: bf16 outputs C against the fp32 oracle R32,

    max_ij |C_ij - R32_ij| / max(|R32_ij|, rms(R32))  <=  2e-2

The floor rms(R32) keeps near-zero outputs (cancellation in long dot products)
from dominating the ratio; a correct kernel lands near the bf16 half-ulp,
2^-9 ~ 1.95e-3, plus a small fp32 reordering error.
"""
from __future__ import annotations

import numpy as np

REL_TOL = 2e-2


def bf16_bits_to_f64(h) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def rel_err(C_bits, R32) -> float:
    C = bf16_bits_to_f64(C_bits)
    R = np.asarray(R32, dtype=np.float64)
    if R.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(R * R)))
    floor = np.maximum(np.abs(R), rms if rms > 0 else 1.0)
    return float(np.max(np.abs(C - R) / floor))


def assert_gemm_close(C_bits, R32, tol: float = REL_TOL, what: str = ""):
    e = rel_err(C_bits, R32)
    assert e <= tol, f"{what}: max relative error {e:.3e} > {tol:.1e}"
    return e
