"""Per-XCD latency / affinity probe on the device, through the C ABI.

Absolute latencies are not pinned (the paper gives none for this chip); what
is checked holds on any part with per-XCD L2s and a memory-side cache: the
three regimes order as L2 < memory-side cache < HBM on every XCD, the groups
partition the XCDs, home shares and the unclassified share add up to one, and
the oracle's analysis of the measured HBM latencies equals the library's.
"""
import numpy as np
import pytest

import paper_2609_24270_amd as asym
from oracle import affinity as oaff

pytestmark = pytest.mark.gpu

SMALL = dict(alloc_bytes=4 << 30, n_samples=2048, passes=2, l2_samples=1024, seed=5)


@pytest.fixture(scope="module")
def probe():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    asym.load_library()
    summ, raw = asym.latency_probe(0, want_raw=True, **SMALL)
    print({k: summ[k] for k in ("timer_overhead", "clock_mhz", "l2_hit", "mall_hit", "hbm",
                                "group_of_xcd", "home_share", "unclassified_share")})
    print("hbm_by_home", [[round(v, 1) for v in r] for r in summ["hbm_by_home"]])
    print("corr", [[round(v, 2) for v in r] for r in summ["corr"]])
    return summ, raw


def test_regimes_order_on_every_xcd(probe):
    s, raw = probe
    n_x = s["n_xcds"]
    assert n_x == asym.device_query(0)["n_xccs"]
    assert raw.shape == (3, n_x, SMALL["n_samples"])
    assert (raw[0, :, SMALL["l2_samples"]:] == 0).all()
    assert (raw[0, :, :SMALL["l2_samples"]] > 0).all() and (raw[1:] > 0).all()
    for x in range(n_x):
        assert s["timer_overhead"] < s["l2_hit"][x] < s["mall_hit"][x] < s["hbm"][x], x
    assert 100.0 < s["clock_mhz"] < 5000.0


def test_groups_partition_and_shares(probe):
    s, _ = probe
    g = s["group_of_xcd"]
    assert sorted(set(g)) == list(range(s["n_groups"]))
    assert abs(sum(s["home_share"]) + s["unclassified_share"] - 1.0) < 1e-12


def test_oracle_analysis_of_measured_latencies(probe):
    s, raw = probe
    ref = oaff.analyze(raw[2].tolist(), 0.5, 20.0)
    assert s["group_of_xcd"] == ref["group_of_xcd"]
    assert s["home_share"] == ref["home_share"]
    assert s["unclassified_share"] == ref["unclassified_share"]
    assert np.allclose(s["corr"], ref["corr"], atol=1e-12, rtol=0)
    assert np.allclose(s["hbm_by_home"], ref["hbm_by_home"], atol=1e-9, rtol=0)
    # per-regime means are the means of the returned minima
    for x in range(s["n_xcds"]):
        assert s["l2_hit"][x] == pytest.approx(raw[0, x, :SMALL["l2_samples"]].mean(), abs=1e-9)
        assert s["mall_hit"][x] == pytest.approx(raw[1, x].mean(), abs=1e-9)
        assert s["hbm"][x] == pytest.approx(raw[2, x].mean(), abs=1e-9)


def test_probe_rejects_bad_parameters():
    with pytest.raises(asym.AsymError) as e:
        asym.latency_probe(0, n_samples=0)
    assert e.value.status == asym.EINVAL
    with pytest.raises(asym.AsymError):
        asym.latency_probe(0, passes=65)
    with pytest.raises(asym.AsymError):
        asym.latency_probe(0, l2_samples=9000, n_samples=10000)
    with pytest.raises(asym.AsymError):
        asym.latency_probe(0, alloc_bytes=1 << 20)


def test_topology_with_latency_and_affinity_aligned_sets():
    """The full probe keeps the affinity groups in the map; an affinity-aligned
    CU set of half the chip is one whole group."""
    topo = asym.probe_topology(0, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP | asym.PROBE_LATENCY)
    info = topo.info()
    L = topo.latency()
    assert info["group_of_xcd"] == L["group_of_xcd"]
    assert L["passes"] == 8 and L["n_samples"] == 16384
    j = topo.json()
    assert j["latency"]["group_of_xcd"] == L["group_of_xcd"]
    g = L["group_of_xcd"]
    sizes = [g.count(k) for k in range(L["n_groups"])]
    print("groups", g, "sizes", sizes, "home", L["home_share"])
    n_x = info["n_xcds"]
    per_xcd = info["cus_per_xcd"][0]
    if sizes and max(sizes) * per_xcd <= info["n_cus"] and all(c == per_xcd for c in info["cus_per_xcd"]):
        n = sizes[0] * per_xcd
        bits = topo.cuset(n, asym.CUSET_AFFINITY_ALIGNED)
        counts = topo.cuset_counts(bits)
        xs = [x for x in range(n_x) if counts[x]]
        assert all(counts[x] == per_xcd for x in xs)
        assert len({g[x] for x in xs}) == 1, (xs, g)
