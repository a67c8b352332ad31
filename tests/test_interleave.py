"""Partition-hash discovery: pins for the oracle, then the library's host
analysis against the oracle (no GPU).

The oracle is pinned to structures planted in synthetic latencies: a parity
over chosen bits inside a translation page with a random bit per page above it
(the bits it must recover, the bits it must call undetermined, the
granularity), a map that is not one parity, a hand-counted case, untested bits,
and inputs where no address has a home.
"""
import numpy as np
import pytest

import paper_2609_24270_amd as asym
from oracle import interleave as oil
from paper_2609_24270_amd import workloads

LO, HI = 7, 30


def _run(seed, mask, rule="xor", page_bits=21, n_bases=64, n_pairs=4):
    offs, block = workloads.interleave_layout(seed, n_bases, LO, HI, n_pairs)
    L, home = workloads.planted_interleave_latency(seed + 1, offs, mask, page_bits, rule)
    return offs, block, L, home, oil.analyze(L.tolist(), offs, block)


def test_oracle_recovers_a_planted_parity_inside_the_page():
    mask = (1 << 12) | (1 << 15) | (1 << 18) | (1 << 24)   # bit 24 is above the 2 MiB page
    offs, block, L, home, r = _run(3, mask)
    assert r["home"] == home
    assert r["group_of_xcd"] == [0, 0, 0, 0, 1, 1, 1, 1]
    for b in range(LO, 21):
        assert r["verdict"][b] == (1 if (mask >> b) & 1 else 0), b
        assert r["flip_fraction"][b] == float((mask >> b) & 1)
        assert r["usable"][b] == 64
    # above the page the per-page bit makes every flip a coin toss
    assert all(r["verdict"][b] == oil.UNDETERMINED for b in range(21, HI))
    assert r["hash_mask"] == mask & ((1 << 21) - 1)
    assert r["lowest_bit"] == 12 and r["granularity"] == 4096
    assert r["determined_below"] == 21
    assert r["pair_checks"] > 0 and r["linear_consistency"] == 1.0
    assert all(r["verdict"][b] == oil.NOT_TESTED for b in list(range(LO)) + list(range(HI, 64)))


def test_oracle_with_contiguous_pages_sees_every_bit():
    mask = (1 << 9) | (1 << 13) | (1 << 22) | (1 << 27)
    _, _, _, _, r = _run(5, mask, page_bits=40)
    assert r["hash_mask"] == mask
    assert r["determined_below"] == HI
    assert r["lowest_bit"] == 9 and r["granularity"] == 512
    assert r["linear_consistency"] == 1.0 and r["pair_checks"] == 64 * 4


def test_oracle_flags_a_map_that_is_not_one_parity():
    """home = b12 XOR (b13 AND b14): bit 12 always flips it, bits 13 and 14 about
    half of the time, so they are undetermined and the granularity stands on
    the bits below 13."""
    mask = (1 << 12) | (1 << 13) | (1 << 14)
    _, _, _, _, r = _run(7, mask, rule="mixed", n_bases=200)
    assert r["verdict"][12] == 1
    assert r["verdict"][13] == oil.UNDETERMINED and r["verdict"][14] == oil.UNDETERMINED
    assert 0.3 < r["flip_fraction"][13] < 0.7 and 0.3 < r["flip_fraction"][14] < 0.7
    assert r["determined_below"] == 13
    assert r["lowest_bit"] == 12 and r["granularity"] == 4096


def test_oracle_counts_by_hand():
    """Three blocks (base, base^bit7, base^bit8, base^bit7^bit8) with homes set
    by hand: bit 7 flips the home in 2 of 3 blocks, bit 8 in all 3."""
    homes = [0, 1, 1, 0,
             1, 0, 0, 1,
             0, 0, 1, 1]
    offs = []
    for base in (0x10000, 0x20000, 0x30000):
        offs += [base, base ^ 0x80, base ^ 0x100, base ^ 0x180]
    L = [[735 + (215 if h != (x >= 4) else 0) + x for h in homes] for x in range(8)]
    r = oil.analyze(L, offs, 4)
    assert r["home"] == homes
    assert r["usable"][7] == 3 and abs(r["flip_fraction"][7] - 2 / 3) < 1e-15
    assert r["verdict"][7] == oil.UNDETERMINED
    assert r["usable"][8] == 3 and r["flip_fraction"][8] == 1.0 and r["verdict"][8] == 1
    # pairs need both verdicts: bit 7 has none, so no pair is counted
    assert r["pair_checks"] == 0 and r["linear_consistency"] == -1.0
    assert r["determined_below"] == 7 and r["granularity"] == -1


def test_oracle_without_homes_decides_nothing():
    offs, block = workloads.interleave_layout(9, 8, LO, 12, 1)
    L = [[800] * len(offs) for _ in range(8)]
    r = oil.analyze(L, offs, block)
    assert r["unclassified_share"] == 1.0
    assert all(r["verdict"][b] == oil.UNDETERMINED for b in range(LO, 12))
    assert r["hash_mask"] == 0 and r["lowest_bit"] == -1 and r["granularity"] == -1


def test_oracle_rejects_partial_blocks():
    with pytest.raises(ValueError):
        oil.analyze([[1, 2, 3]] * 8, [0, 128, 256], 2)
