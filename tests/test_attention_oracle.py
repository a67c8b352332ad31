"""Pins for the decode-attention oracle (CPU only).

Each pin is a fact of the mathematics, not the oracle's formula retyped: a
single token returns its value row; identical keys average the values; a key
far ahead of the rest returns its value row; two tokens give the logistic
weight in closed form; token order does not matter; query head h reads
key/value head h // (H_q / H_kv) (planted per-head constant values); scaling
q by c and the scale by 1/c changes nothing; the log-sum-exp of identical
scores is s + log S_k.
"""
import math

import numpy as np
import pytest

from oracle import attention as oat
from oracle import f32_to_bf16


def bf(x):
    return f32_to_bf16(np.asarray(x, dtype=np.float32))


def rnd(shape, seed, sigma=1.0):
    return bf(np.random.default_rng(seed).normal(0, sigma, shape))


def test_one_token_returns_its_value_row():
    q, k, v = rnd((2, 4, 128), 1), rnd((2, 2, 1, 128), 2), rnd((2, 2, 1, 128), 3)
    O, lse = oat.decode_attention(q, k, v, 0.1)
    V = oat.bf16_to_f64(v)
    for b in range(2):
        for h in range(4):
            assert np.array_equal(O[b, h], V[b, h // 2, 0])
            s = 0.1 * float(oat.bf16_to_f64(q)[b, h] @ oat.bf16_to_f64(k)[b, h // 2, 0])
            assert abs(lse[b, h] - s) < 1e-12 * max(1.0, abs(s))


def test_identical_keys_average_the_values():
    S = 37
    q = rnd((1, 1, 128), 4)
    krow = rnd((128,), 5)
    k = np.tile(krow, (1, 1, S, 1))
    v = rnd((1, 1, S, 128), 6)
    O, lse = oat.decode_attention(q, k, v, 1 / math.sqrt(128))
    V = oat.bf16_to_f64(v)[0, 0]
    assert np.allclose(O[0, 0], V.mean(axis=0), rtol=0, atol=1e-13)
    s = float(oat.bf16_to_f64(q)[0, 0] @ oat.bf16_to_f64(krow)) / math.sqrt(128)
    assert abs(lse[0, 0] - (s + math.log(S))) < 1e-12


def test_dominant_key_returns_its_value_row():
    S, t = 64, 23
    q = bf(np.ones((1, 1, 128)))
    k = np.zeros((1, 1, S, 128), dtype=np.float32)
    k[0, 0, t] = 1.0          # score 128 * scale ahead of every other key's 0
    v = rnd((1, 1, S, 128), 7)
    O, _ = oat.decode_attention(q, bf(k), v, 1.0)
    V = oat.bf16_to_f64(v)[0, 0]
    # the other 63 weights are each e^-128 of the top one
    assert np.allclose(O[0, 0], V[t], rtol=0, atol=64 * math.exp(-128) * np.abs(V).max())


def test_two_tokens_logistic_closed_form():
    q = bf(np.full((1, 1, 128), 0.5))
    k = np.zeros((1, 1, 2, 128), dtype=np.float32)
    k[0, 0, 0, :8] = 1.0        # s0 = 8 * 0.5 * scale
    k[0, 0, 1, :3] = -1.0       # s1 = -3 * 0.5 * scale
    v = rnd((1, 1, 2, 128), 8)
    scale = 0.25
    O, lse = oat.decode_attention(q, bf(k), v, scale)
    s0, s1 = 8 * 0.5 * scale, -3 * 0.5 * scale
    w0 = 1.0 / (1.0 + math.exp(s1 - s0))
    V = oat.bf16_to_f64(v)[0, 0]
    assert np.allclose(O[0, 0], w0 * V[0] + (1 - w0) * V[1], rtol=0, atol=1e-15)
    assert abs(lse[0, 0] - math.log(math.exp(s0) + math.exp(s1))) < 1e-14


def test_token_order_does_not_matter():
    q, k, v = rnd((3, 8, 128), 9), rnd((3, 2, 50, 128), 10), rnd((3, 2, 50, 128), 11)
    perm = np.random.default_rng(12).permutation(50)
    O1, l1 = oat.decode_attention(q, k, v, 0.088)
    O2, l2 = oat.decode_attention(q, k[:, :, perm], v[:, :, perm], 0.088)
    assert np.allclose(O1, O2, rtol=0, atol=1e-12) and np.allclose(l1, l2, rtol=0, atol=1e-12)


@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (32, 8), (6, 6), (16, 1)])
def test_query_head_reads_kv_head_h_over_group(Hq, Hkv):
    S = 9
    q, k = rnd((2, Hq, 128), 13), rnd((2, Hkv, S, 128), 14)
    v = np.zeros((2, Hkv, S, 128), dtype=np.float32)
    for g in range(Hkv):
        v[:, g] = g + 1          # every value row of key/value head g is g + 1
    O, _ = oat.decode_attention(q, k, bf(v), 0.1)
    G = Hq // Hkv
    for h in range(Hq):
        assert np.allclose(O[:, h], h // G + 1, rtol=0, atol=1e-12)


def test_scale_moves_between_query_and_scale():
    q, k, v = rnd((1, 4, 128), 15), rnd((1, 4, 30, 128), 16), rnd((1, 4, 30, 128), 17)
    O1, l1 = oat.decode_attention(q, k, v, 0.125)
    q2 = bf(oat.bf16_to_f64(q) * 2.0)       # exact: a power of two
    O2, l2 = oat.decode_attention(q2, k, v, 0.0625)
    assert np.allclose(O1, O2, rtol=0, atol=1e-12) and np.allclose(l1, l2, rtol=0, atol=1e-12)


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oat.decode_attention(rnd((1, 3, 128), 1), rnd((1, 2, 4, 128), 2), rnd((1, 2, 4, 128), 3), 1.0)
    with pytest.raises(ValueError):
        oat.decode_attention(rnd((1, 2, 128), 1), rnd((1, 2, 4, 64), 2), rnd((1, 2, 4, 64), 3), 1.0)
