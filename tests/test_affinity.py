"""Affinity analysis: pins for the oracle, then the library's host analysis
against the oracle (no GPU).

The oracle is pinned to facts outside itself: numpy's correlation routine,
planted structures it must recover (Appendix G's MI300X picture of four XCD
pairs with three tiers, and a two-halves layout), transitivity of grouping,
the tie margin at its boundary, and constant inputs.
"""
import numpy as np
import pytest

import paper_2609_24270_amd as asym
from oracle import affinity as oaff
from paper_2609_24270_amd import workloads


def test_pearson_matches_numpy():
    rng = np.random.default_rng(7)
    for n in (2, 3, 17, 1000):
        u = rng.integers(600, 1000, n)
        v = (u * 0.3 + rng.integers(0, 100, n)).astype(np.int64)
        want = float(np.corrcoef(u.astype(float), v.astype(float))[0, 1])
        assert abs(oaff.pearson(list(u), list(v)) - want) < 1e-12
    # perfectly (anti-)correlated rows
    u = list(range(50))
    assert abs(oaff.pearson(u, [3 * a + 5 for a in u]) - 1.0) < 1e-15
    assert abs(oaff.pearson(u, [-2 * a for a in u]) + 1.0) < 1e-15
    # a constant row has no correlation
    assert oaff.pearson([5] * 10, list(range(10))) == 0.0


def test_oracle_recovers_four_pairs_three_tiers():
    """Appendix G: XCD pairs {0,1},{2,3},{4,5},{6,7}, each homing ~25% of the
    addresses, local / adjacent / opposite tiers about 110 and 219 cycles apart."""
    L, home = workloads.planted_latency(11, 4000)
    r = oaff.analyze(L.tolist(), 0.5, 20.0)
    assert r["group_of_xcd"] == [0, 0, 1, 1, 2, 2, 3, 3]
    assert r["n_groups"] == 4
    assert r["unclassified_share"] == 0.0
    assert r["home"] == list(home)
    for s in r["home_share"]:
        assert abs(s - 0.25) < 4 * np.sqrt(0.25 * 0.75 / 4000)
    # tiers seen from XCD 0: own group, two adjacent groups, the opposite one
    t = r["hbm_by_home"][0]
    mean_extra = (40 - 1) / 2 + (12 - 1) / 2  # common offset + jitter
    for g, tier in zip(range(4), (707, 817, 817, 926)):
        assert abs(t[g] - tier - mean_extra) < 3.0
    # correlation: ~1 within a pair, 0 to adjacent, -1 to opposite pairs
    c = r["corr"]
    assert c[0][1] > 0.95 and abs(c[0][2]) < 0.1 and c[0][6] < -0.9


def test_oracle_recovers_two_halves():
    grp = (0, 0, 0, 0, 1, 1, 1, 1)
    L, home = workloads.planted_latency(12, 3000, grp=grp, dist=((0, 1), (1, 0)), tiers=(700, 800))
    r = oaff.analyze(L.tolist())
    assert r["group_of_xcd"] == list(grp)
    assert r["home"] == list(home)
    assert abs(sum(r["home_share"]) - 1.0) < 1e-12


def test_oracle_grouping_is_transitive():
    # 0~1 and 1~2 above the threshold, 0~2 below it: one group of three
    corr = [[1, .9, .1, 0], [.9, 1, .8, 0], [.1, .8, 1, 0], [0, 0, 0, 1]]
    assert oaff.groups_from_corr(corr, 0.5) == ([0, 0, 0, 1], 2)
    # exactly at the threshold does not join
    assert oaff.groups_from_corr([[1, .5], [.5, 1]], 0.5) == ([0, 1], 2)


def _tie_rows(n=64):
    """Two anti-correlated pairs whose group means differ by 20 cycles on even
    addresses and by 0 on odd ones."""
    s = np.arange(n) % 2
    a = 700 + 10 * s
    b = 720 - 10 * s
    return np.stack([a, a, b, b]).astype(np.int64)


def test_oracle_tie_margin_boundary():
    L = _tie_rows().tolist()
    r = oaff.analyze(L, 0.5, 20.0)
    assert r["group_of_xcd"] == [0, 0, 1, 1]
    # a gap of 20 is not below a margin of 20 (classified); a gap of 0 is
    assert r["unclassified_share"] == 0.5 and r["home_share"] == [0.5, 0.0]
    assert oaff.analyze(L, 0.5, 21.0)["unclassified_share"] == 1.0
    # margin 0: equal means go to the lower group
    r = oaff.analyze(L, 0.5, 0.0)
    assert r["unclassified_share"] == 0.0 and r["home_share"] == [1.0, 0.0]


def test_oracle_constant_rows_stay_apart():
    L = [[800] * 32 for _ in range(4)]
    r = oaff.analyze(L, 0.5, 20.0)
    assert r["group_of_xcd"] == [0, 1, 2, 3]
    assert r["unclassified_share"] == 1.0


# -- the library's host analysis against the oracle ------------------------

def _compare(lib, ref):
    assert lib["group_of_xcd"] == ref["group_of_xcd"]
    assert lib["n_groups"] == ref["n_groups"]
    assert lib["home_share"] == pytest.approx(ref["home_share"], abs=0)
    assert lib["unclassified_share"] == ref["unclassified_share"]
    assert np.allclose(lib["corr"], ref["corr"], atol=1e-12, rtol=0)
    assert np.allclose(lib["hbm"], ref["hbm"], atol=1e-9, rtol=0)
    assert np.allclose(lib["hbm_by_home"], ref["hbm_by_home"], atol=1e-9, rtol=0)


@pytest.mark.parametrize("case", ["pairs", "halves", "noise", "one_xcd", "tie"])
def test_library_analysis_matches_oracle(case):
    thr, tie = 0.5, 20.0
    if case == "pairs":
        L, _ = workloads.planted_latency(21, 2048)
    elif case == "halves":
        L, _ = workloads.planted_latency(22, 999, grp=(0, 0, 0, 0, 1, 1, 1, 1),
                                         dist=((0, 1), (1, 0)), tiers=(700, 800))
    elif case == "noise":   # no structure: many small groups, many ties
        L = np.random.default_rng(23).integers(700, 760, (8, 500)).astype(np.uint32)
    elif case == "one_xcd":
        L = np.random.default_rng(24).integers(700, 900, (1, 100)).astype(np.uint32)
    else:
        L = _tie_rows(80).astype(np.uint32)
    lib = asym.latency_analyze(L, thr, tie)
    ref = oaff.analyze(L.tolist(), thr, tie)
    _compare(lib, ref)
    assert lib["passes"] == -1 and lib["timer_overhead"] == -1.0


def test_library_analysis_rejects_bad_input():
    with pytest.raises(asym.AsymError) as e:
        asym.latency_analyze(np.zeros((17, 4), dtype=np.uint32))
    assert e.value.status == asym.EINVAL
    with pytest.raises(asym.AsymError):
        asym.latency_analyze(np.zeros((2, 4), dtype=np.uint32), tie_cycles=-1.0)
    with pytest.raises(ValueError):
        asym.latency_analyze(np.zeros(4, dtype=np.uint32))


def test_latency_params_defaults():
    p = asym.latency_params()
    assert (p.alloc_bytes, p.n_samples, p.passes, p.l2_samples, p.seed) == (0, 16384, 8, 4096, 0)
    assert p.group_threshold == 0.5 and p.tie_cycles == 20.0
    with pytest.raises(TypeError):
        asym.latency_params(bogus=1)
