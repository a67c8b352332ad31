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
    # planted tiers 735 / 950 plus offsets in [0, 40) and jitter in [0, 12)
    assert 735 <= r["local_cycles"] < 735 + 51 and 950 <= r["remote_cycles"] < 950 + 51


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


def _lib_result(L, offs, block, threshold=0.5, tie=20.0, decide=0.1):
    lib = asym.load_library()
    return asym.interleave_analyze(np.asarray(L, dtype=np.uint32), offs, block, threshold, tie, decide)


def _compare(res, ref):
    for k in ("n_groups", "group_of_xcd", "home", "usable", "verdict", "hash_mask", "lowest_bit",
              "determined_below", "granularity", "pair_checks", "pair_agree"):
        assert res[k] == ref[k], k
    for k in ("flip_fraction",):
        assert all(abs(a - b) < 1e-12 for a, b in zip(res[k], ref[k])), k
    for k in ("linear_consistency", "unclassified_share", "local_cycles", "remote_cycles"):
        assert abs(res[k] - ref[k]) < 1e-9 * max(1.0, abs(ref[k])), k


@pytest.mark.parametrize("case", ["xor_page", "contiguous", "mixed", "no_homes", "one_bit"])
def test_library_analysis_matches_oracle(case):
    if case == "xor_page":
        offs, block = workloads.interleave_layout(3, 64, LO, HI, 4)
        L, _ = workloads.planted_interleave_latency(4, offs, (1 << 12) | (1 << 15) | (1 << 24))
    elif case == "contiguous":
        offs, block = workloads.interleave_layout(5, 32, LO, 24, 6)
        L, _ = workloads.planted_interleave_latency(6, offs, (1 << 8) | (1 << 22), page_bits=40)
    elif case == "mixed":
        offs, block = workloads.interleave_layout(7, 100, LO, 20, 3)
        L, _ = workloads.planted_interleave_latency(8, offs, (1 << 12) | (1 << 13) | (1 << 14), rule="mixed")
    elif case == "no_homes":
        offs, block = workloads.interleave_layout(9, 8, LO, 12, 1)
        L = np.full((8, len(offs)), 800, dtype=np.uint32)
    else:
        offs, block = workloads.interleave_layout(10, 16, 12, 13, 0)
        L, _ = workloads.planted_interleave_latency(11, offs, 1 << 12)
    ref = oil.analyze(np.asarray(L).tolist(), offs, block)
    _compare(_lib_result(L, offs, block), ref)


def test_library_analysis_rejects_bad_input():
    offs, block = workloads.interleave_layout(3, 4, LO, 10, 1)
    L = np.full((8, len(offs)), 800, dtype=np.uint32)
    with pytest.raises(asym.AsymError):
        asym.interleave_analyze(L[:, :-1], offs[:-1], block)     # partial block
    with pytest.raises(asym.AsymError):
        asym.interleave_analyze(L, offs, block, decide=0.5)      # margin out of range
    with pytest.raises(asym.AsymError):
        asym.interleave_analyze(np.full((17, len(offs)), 800, dtype=np.uint32), offs, block)


def test_interleave_params_defaults():
    p = asym.interleave_params_default()
    assert (p["n_bases"], p["lo_bit"], p["hi_bit"], p["n_pairs"], p["passes"]) == (128, 7, 32, 4, 8)
    assert p["decide"] == 0.1 and p["tie_cycles"] == 20.0 and p["group_threshold"] == 0.5
