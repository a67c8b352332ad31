"""Oracle for decode attention with grouped key/value heads.  TEST INFRASTRUCTURE ONLY.

Section 7.1 runs attention kernels (multi-head and grouped-query attention) as
full-GPU workloads, decode being one query token per request against a cached
key/value sequence (Appendix F: S_q = 1, head dimension 128, 32 key/value
heads for multi-head and 8 for grouped-query attention).  What the kernel
computes is the plain definition, written out here in float64 with numpy:

    for request b and query head h, with key/value head g = h // (H_q / H_kv):
        s_t = scale * <q[b, h], K[b, g, t]>          t = 0 .. S_k - 1
        p_t = exp(s_t - max_t s_t) / sum_t exp(s_t - max_t s_t)
        O[b, h] = sum_t p_t V[b, g, t]
        lse[b, h] = max_t s_t + log(sum_t exp(s_t - max_t s_t))

No blocking, no split of the sequence, no online rescaling: one softmax over
the whole sequence per (request, head).  Inputs are bf16 bit patterns (uint16),
widened exactly to float64.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def decode_attention(q_bits, k_bits, v_bits, scale: float):
    """q: uint16 [B, H_q, D]; k, v: uint16 [B, H_kv, S_k, D].
    Returns (O float64 [B, H_q, D], lse float64 [B, H_q])."""
    q = bf16_to_f64(q_bits)
    k = bf16_to_f64(k_bits)
    v = bf16_to_f64(v_bits)
    B, Hq, D = q.shape
    Bk, Hkv, S, Dk = k.shape
    if Bk != B or Dk != D or v.shape != k.shape or Hq % Hkv or S < 1:
        raise ValueError("shapes: q [B, H_q, D], k and v [B, H_kv, S_k, D], H_kv divides H_q, S_k >= 1")
    G = Hq // Hkv
    O = np.zeros((B, Hq, D))
    lse = np.zeros((B, Hq))
    for b in range(B):
        for h in range(Hq):
            g = h // G
            s = scale * (k[b, g] @ q[b, h])
            m = s.max()
            e = np.exp(s - m)
            tot = e.sum()
            O[b, h] = (e / tot) @ v[b, g]
            lse[b, h] = m + np.log(tot)
    return O, lse
