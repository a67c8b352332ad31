"""Partition-hash discovery on the device, through the C ABI.

The chip's hash has no pinned value (the paper dissects NVIDIA parts only), so
what is checked is: the probe lays its blocks out as documented, the oracle's
analysis of the measured latencies equals the library's in every field, the
walked range starts on a 2 MiB boundary, and two runs with different bases
agree on every bit both of them decide.  The verdicts themselves are printed.
"""
import numpy as np
import pytest

import paper_2609_24270_amd as asym
from oracle import interleave as oil

pytestmark = pytest.mark.gpu

RUN = dict(n_bases=96, lo_bit=7, hi_bit=30, n_pairs=4, passes=4)


def _summary(r):
    bits = {b: (r["verdict"][b], round(r["flip_fraction"][b], 3)) for b in range(RUN["lo_bit"], RUN["hi_bit"])}
    return {"hash_mask": hex(r["hash_mask"]), "lowest_bit": r["lowest_bit"],
            "granularity": r["granularity"], "determined_below": r["determined_below"],
            "linear": (r["pair_agree"], r["pair_checks"]), "groups": r["group_of_xcd"],
            "unclassified": round(r["unclassified_share"], 4),
            "local/remote": (round(r["local_cycles"], 1), round(r["remote_cycles"], 1)),
            "base_align": hex(r["base_align"]), "bits": bits}


@pytest.fixture(scope="module")
def runs():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    asym.load_library()
    out = []
    for seed in (1, 2):
        r, offs, lat, home = asym.interleave_probe(0, seed=seed, **RUN)
        print(f"seed {seed}:", _summary(r), flush=True)
        out.append((r, offs, lat, home))
    return out


def test_layout_is_as_documented(runs):
    lo, hi, npair = RUN["lo_bit"], RUN["hi_bit"], RUN["n_pairs"]
    block = 1 + hi - lo + npair
    for r, offs, lat, home in runs:
        assert r["block"] == block and r["n_addresses"] == RUN["n_bases"] * block == len(offs)
        o = [int(v) for v in offs]
        for b0 in range(0, len(o), block):
            base = o[b0]
            assert base % 128 == 0 and base < (1 << hi)
            assert o[b0 + 1: b0 + 1 + hi - lo] == [base ^ (1 << k) for k in range(lo, hi)]
            for v in o[b0 + 1 + hi - lo: b0 + block]:
                d = v ^ base
                assert bin(d).count("1") == 2 and d >> lo << lo == d and d < (1 << hi)
        assert r["base_align"] >= (2 << 20) and r["base_align"] & (r["base_align"] - 1) == 0
        assert lat.shape == (r["n_xcds"], len(offs)) and (lat > 0).all()


def test_library_analysis_matches_the_oracle_on_measured_latencies(runs):
    block = 1 + RUN["hi_bit"] - RUN["lo_bit"] + RUN["n_pairs"]
    for r, offs, lat, home in runs:
        ref = oil.analyze(lat.tolist(), [int(v) for v in offs], block)
        assert [int(h) for h in home] == ref["home"]
        for k in ("n_groups", "usable", "verdict", "hash_mask", "lowest_bit", "determined_below",
                  "granularity", "pair_checks", "pair_agree"):
            assert r[k] == ref[k], k
        assert r["group_of_xcd"] == ref["group_of_xcd"]
        assert all(abs(a - b) < 1e-12 for a, b in zip(r["flip_fraction"], ref["flip_fraction"]))
        for k in ("linear_consistency", "unclassified_share", "local_cycles", "remote_cycles"):
            assert abs(r[k] - ref[k]) < 1e-9 * max(1.0, abs(ref[k])), k


def test_two_runs_agree_where_both_decide(runs):
    (r1, *_), (r2, *_) = runs
    both = [b for b in range(64) if r1["verdict"][b] in (0, 1) and r2["verdict"][b] in (0, 1)]
    assert [r1["verdict"][b] for b in both] == [r2["verdict"][b] for b in both]
    assert r1["group_of_xcd"] == r2["group_of_xcd"]


def test_probe_rejects_bad_parameters():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    for bad in (dict(lo_bit=6), dict(hi_bit=37), dict(lo_bit=20, hi_bit=20), dict(n_bases=0),
                dict(n_pairs=65), dict(passes=0), dict(decide=0.5), dict(lo_bit=20, hi_bit=21, n_pairs=1)):
        with pytest.raises(asym.AsymError):
            asym.interleave_probe(0, **{**RUN, **bad})
