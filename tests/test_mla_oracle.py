"""Pins for the MLA decode oracle (CPU only).

Each pin is a fact of the mathematics of latent attention, not the oracle's
formula retyped: one token returns its latent row; identical rows average to
that row (the value is the key's latent part, so averaging identical rows
returns it) with lse = s + log S_k; equal latent parts with different rotary
parts return the latent whatever the weights, while the rotary part alone
sets the weights (two tokens: the logistic weight in closed form); a row far
ahead of the others returns its latent; token order does not matter; the
value is the first 512 values of the row, never the rotary tail; heads are
independent; the scale can move into q.
"""
import math

import numpy as np
import pytest

from oracle import f32_to_bf16
from oracle import mla


def bf(x):
    return f32_to_bf16(np.asarray(x, dtype=np.float32))


def rnd(shape, seed, sigma=1.0):
    return bf(np.random.default_rng(seed).normal(0, sigma, shape))


def test_one_token_returns_its_latent_row():
    q, kv = rnd((2, 16, 576), 1), rnd((2, 1, 576), 2)
    O, lse = mla.mla_decode(q, kv, 0.07)
    Q, KV = mla.bf16_to_f64(q), mla.bf16_to_f64(kv)
    for b in range(2):
        for h in range(16):
            assert np.array_equal(O[b, h], KV[b, 0, :512])
            s = 0.07 * float(Q[b, h] @ KV[b, 0])
            assert abs(lse[b, h] - s) < 1e-12 * max(1.0, abs(s))


def test_identical_rows_and_the_log_sum_exp():
    S = 45
    q = rnd((1, 3, 576), 3)
    row = rnd((576,), 4)
    kv = np.tile(row, (1, S, 1))
    O, lse = mla.mla_decode(q, kv, 1 / math.sqrt(576))
    R = mla.bf16_to_f64(row)
    for h in range(3):
        assert np.allclose(O[0, h], R[:512], rtol=0, atol=1e-13)
        s = float(mla.bf16_to_f64(q)[0, h] @ R) / math.sqrt(576)
        assert abs(lse[0, h] - (s + math.log(S))) < 1e-12


def test_rotary_part_sets_the_weights_latent_part_sets_the_values():
    # two tokens with the same latent part: the output is that latent for any
    # weights; with zero latent parts in q only the rotary dot products
    # remain, and the two-token weight is the logistic of their difference
    lat = rnd((512,), 5)
    r0, r1 = rnd((64,), 6), rnd((64,), 7)
    kv = np.zeros((1, 2, 576), dtype=np.uint16)
    kv[0, 0, :512] = lat
    kv[0, 1, :512] = lat
    kv[0, 0, 512:] = r0
    kv[0, 1, 512:] = r1
    q = np.zeros((1, 1, 576), dtype=np.uint16)
    q[0, 0, 512:] = rnd((64,), 8)
    O, lse = mla.mla_decode(q, kv, 0.5)
    L = mla.bf16_to_f64(lat)
    assert np.allclose(O[0, 0], L, rtol=0, atol=1e-13)
    Q = mla.bf16_to_f64(q)[0, 0, 512:]
    s0 = 0.5 * float(Q @ mla.bf16_to_f64(r0))
    s1 = 0.5 * float(Q @ mla.bf16_to_f64(r1))
    assert abs(lse[0, 0] - (max(s0, s1) + math.log1p(math.exp(-abs(s0 - s1))))) < 1e-12
    # distinct latents: O = w0 * lat0 + w1 * lat1 with w1 = logistic(s1 - s0)
    lat1 = rnd((512,), 9)
    kv[0, 1, :512] = lat1
    O, _ = mla.mla_decode(q, kv, 0.5)
    w1 = 1.0 / (1.0 + math.exp(s0 - s1))
    want = (1 - w1) * L + w1 * mla.bf16_to_f64(lat1)
    assert np.allclose(O[0, 0], want, rtol=0, atol=1e-12)


def test_value_is_the_latent_part_not_the_rotary_tail():
    # rotary tails of huge magnitude change the weights but never the values
    S = 9
    kv = rnd((1, S, 576), 10).copy()
    big = bf(np.full((64,), 300.0))
    kv[0, :, 512:] = big
    q = np.zeros((1, 2, 576), dtype=np.uint16)
    q[0, :, :512] = rnd((2, 512), 11)
    O, _ = mla.mla_decode(q, kv, 0.05)
    KV = mla.bf16_to_f64(kv)[0]
    lo, hi = KV[:, :512].min(axis=0), KV[:, :512].max(axis=0)
    assert np.all(O[0] >= lo - 1e-12) and np.all(O[0] <= hi + 1e-12)
    assert np.abs(O).max() < 10.0


def test_dominant_row_returns_its_latent():
    S, t = 70, 41
    q = bf(np.ones((1, 1, 576)))
    kv = np.zeros((1, S, 576), dtype=np.float32)
    kv[0, :, :512] = np.random.default_rng(12).normal(0, 1, (S, 512))
    kv[0, :, 512:] = 0.0
    kv[0, t, 512:] = 1.0            # score 64 ahead of every other token's rotary part
    q = q.copy()
    q[0, 0, :512] = 0               # only the rotary part scores
    O, _ = mla.mla_decode(q, bf(kv), 1.0)
    KV = mla.bf16_to_f64(bf(kv))[0]
    assert np.allclose(O[0, 0], KV[t, :512], rtol=0, atol=1e-20 + 1e-25 * S)
    assert np.abs(O[0, 0] - KV[t, :512]).max() < 1e-25


def test_token_order_does_not_matter_and_heads_are_independent():
    q, kv = rnd((2, 32, 576), 13), rnd((2, 50, 576), 14)
    O, lse = mla.mla_decode(q, kv, 1 / math.sqrt(192))
    perm = np.random.default_rng(15).permutation(50)
    O2, lse2 = mla.mla_decode(q, kv[:, perm], 1 / math.sqrt(192))
    assert np.allclose(O, O2, rtol=1e-12, atol=1e-13) and np.allclose(lse, lse2, rtol=1e-13)
    # head 5's output does not depend on the other heads' queries
    q2 = q.copy()
    q2[:, [0, 1, 7, 31]] = rnd((2, 4, 576), 16)
    O3, _ = mla.mla_decode(q2, kv, 1 / math.sqrt(192))
    assert np.array_equal(O3[:, 5], O[:, 5])


def test_scale_moves_into_q():
    q = np.random.default_rng(17).integers(-4, 5, (1, 2, 576)).astype(np.float32)
    kv = rnd((1, 20, 576), 18)
    O1, l1 = mla.mla_decode(bf(q), kv, 0.25)
    O2, l2 = mla.mla_decode(bf(q * 0.25), kv, 1.0)   # exact in bf16 (powers of two)
    assert np.allclose(O1, O2, rtol=1e-13, atol=1e-14) and np.allclose(l1, l2, rtol=1e-13)


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        mla.mla_decode(rnd((1, 1, 512), 0), rnd((1, 3, 576), 1), 1.0)
    with pytest.raises(ValueError):
        mla.mla_decode(rnd((1, 1, 576), 0), rnd((2, 3, 576), 1), 1.0)
