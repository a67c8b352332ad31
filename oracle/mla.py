"""Oracle for multi-head latent attention, decode.  TEST INFRASTRUCTURE ONLY.

Section 7.1 runs multi-head latent attention (MLA) decode as a full-GPU
kernel, and Appendix F counts its working set as one compressed key/value
row of 512 + 64 values per token, shared by every query head.  In the decode
form of MLA (projections absorbed into the query, as in the DeepSeek-V2
design the paper cites), request b caches per token t one row
    Kc[b, t] = [ c_t (512 latent values) ; r_t (64 rotary key values) ]
and every query head h has a 576-wide query q[b, h].  The latent c_t serves
as the value.  What the kernel computes is this definition, in float64 with
numpy:

    s_t = scale * <q[b, h], Kc[b, t]>                 t = 0 .. S_k - 1 (576 terms)
    p_t = exp(s_t - max s) / sum_t exp(s_t - max s)
    O[b, h] = sum_t p_t Kc[b, t, 0:512]
    lse[b, h] = max s + log(sum_t exp(s_t - max s))

One softmax over the whole sequence per (request, head); no blocking, no
split, no online rescaling.  Inputs are bf16 bit patterns (uint16), widened
exactly to float64.
"""
from __future__ import annotations

import numpy as np

D_LATENT = 512   # compressed key/value (the value) per token
D_ROPE = 64      # decoupled rotary key part
D_QK = D_LATENT + D_ROPE


def bf16_to_f64(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def mla_decode(q_bits, kv_bits, scale: float):
    """q: uint16 [B, H_q, 576]; kv: uint16 [B, S_k, 576] (latent 512 then
    rotary 64 per token).  Returns (O float64 [B, H_q, 512], lse float64 [B, H_q])."""
    q = bf16_to_f64(q_bits)
    kv = bf16_to_f64(kv_bits)
    B, Hq, D = q.shape
    Bk, S, Dk = kv.shape
    if D != D_QK or Dk != D_QK or Bk != B or S < 1:
        raise ValueError("shapes: q [B, H_q, 576], kv [B, S_k, 576], S_k >= 1")
    O = np.zeros((B, Hq, D_LATENT))
    lse = np.zeros((B, Hq))
    for b in range(B):
        for h in range(Hq):
            s = scale * (kv[b] @ q[b, h])
            m = s.max()
            e = np.exp(s - m)
            tot = e.sum()
            O[b, h] = (e / tot) @ kv[b, :, :D_LATENT]
            lse[b, h] = m + np.log(tot)
    return O, lse
