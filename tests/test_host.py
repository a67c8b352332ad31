"""Host-side logic of libasym against the oracle, on the CPU (no GPU calls).

Covers: every symbol declared in include/asym.h is exported; the tile
schedule equals the oracle's definition (quotas, order, coverage); the
topology map built from synthetic identity records equals the oracle's map and
rejects maps that break the exact invariants; CU-set policies; argument errors
that the library reports before touching a device.
"""
import os
import random
import re

import numpy as np
import pytest

import paper_2609_24270_amd as asym
from oracle import schedule as osched
from oracle import topology as otopo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return asym.load_library()


def test_exports_every_declared_symbol(lib):
    hdr = open(os.path.join(ROOT, "include", "asym.h")).read()
    declared = set(re.findall(r"^\s*(?:int|void|const char\*)\s+(asym_\w+)\s*\(", hdr, re.M))
    assert declared == set(asym.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert asym.version() >= 1


# -- schedule ------------------------------------------------------------------

def _cases():
    rng = random.Random(1234)
    cases = [(32, 32, [32] * 8), (16, 56, [32] * 8), (16, 16, [32] * 8), (1, 1, [32] * 8),
             (2, 65, [24] * 6 + [0, 0]), (16, 16, [16, 10, 22, 16, 13, 19, 16, 16]),
             (7, 3, [1, 0, 0, 0, 0, 0, 0, 0]), (32, 16, [24] * 8)]
    for _ in range(25):
        n = rng.choice([1, 2, 4, 8])
        slots = [rng.randint(0, 32) for _ in range(n)]
        if sum(slots) == 0:
            slots[0] = 1
        cases.append((rng.randint(1, 40), rng.randint(1, 40), slots))
    return cases


@pytest.mark.parametrize("tm,tn,slots", _cases())
def test_schedule_matches_oracle(lib, tm, tn, slots):
    T = tm * tn
    band = osched.band_cost_choice(tm, max(slots))
    # aware: every band apportioned by Hamilton's method, lists band by band
    # (or whole blocks dealt round-robin where a band is shorter than a round)
    order, off, quota = asym.schedule_build(tm, tn, slots, asym.MAP_AWARE)
    lists = osched.aware_lists_auto(tm, tn, slots)
    assert quota == [len(lst) for lst in lists]
    assert order == [t for lst in lists for t in lst]
    assert off[0] == 0 and all(off[x + 1] - off[x] == quota[x] for x in range(len(slots)))
    assert sorted(order) == list(range(T))                     # every tile exactly once
    W = sum(slots)
    n_bands = -(-tm // band)
    # each band's share is within one tile of exact, so the total within n_bands
    assert all(abs(quota[x] - T * slots[x] / W) < n_bands for x in range(len(slots)))
    assert all(q == 0 for q, s in zip(quota, slots) if s == 0)
    # oblivious grouped: the whole banded walk, placed round-robin
    order_g, _, quota_g = asym.schedule_build(tm, tn, slots, asym.MAP_OBLIVIOUS_GROUPED)
    assert order_g == osched.banded_order(tm, tn, band)
    owner = osched.oblivious_assignment(order_g, slots)
    assert quota_g == [sum(1 for v in owner.values() if v == x) for x in range(len(slots))]
    # oblivious row-major
    order_r, _, _ = asym.schedule_build(tm, tn, slots, asym.MAP_OBLIVIOUS_ROWMAJOR)
    assert order_r == osched.rowmajor_order(tm, tn)


def test_schedule_explicit_band(lib):
    order, _, _ = asym.schedule_build(10, 7, [4] * 8, asym.MAP_OBLIVIOUS_GROUPED, band=3)
    assert order == osched.banded_order(10, 7, 3)
    order, _, _ = asym.schedule_build(10, 7, [4] * 8, asym.MAP_AWARE, band=3)
    assert order == [t for lst in osched.aware_lists(10, 7, [4] * 8, 3) for t in lst]


def test_hamilton_pins():
    # textbook cases of the largest-remainder method
    assert osched.hamilton_quotas(10, [1, 1, 1]) == [4, 3, 3]      # tie to the lowest index
    assert osched.hamilton_quotas(7, [5, 3, 2]) == [4, 2, 1]       # 3.5, 2.1, 1.4 -> 3,2,1 + 1 to the .5
    assert osched.hamilton_quotas(100, [1, 0, 3]) == [25, 0, 75]
    assert osched.hamilton_quotas(5, [0, 0, 2]) == [0, 0, 5]


def test_aware_wave_blocks_are_compact():
    # 8192^3 at 256^2 tiles: 32 tiles per XCD per wave form 8 rows x 4 columns,
    # and in each wave all XCDs share the same 8 rows of A
    order, off, quota = asym.schedule_build(32, 32, [32] * 8, asym.MAP_AWARE)
    for w in range(4):
        band_rows = set()
        for x in range(8):
            wave = order[off[x] + 32 * w: off[x] + 32 * (w + 1)]
            rows = {t // 32 for t in wave}
            cols = {t % 32 for t in wave}
            assert len(rows) + len(cols) == 12
            band_rows |= rows
        assert len(band_rows) == 8
    # the grouped-oblivious order spreads each wave over 1 row x 32 columns per XCD
    order_g, _, _ = asym.schedule_build(32, 32, [32] * 8, asym.MAP_OBLIVIOUS_GROUPED)
    own = osched.oblivious_assignment(order_g, [32] * 8)
    first_wave = order_g[:256]
    for x in range(8):
        mine = [t for t in first_wave if own[t] == x]
        assert len({t // 32 for t in mine}) + len({t % 32 for t in mine}) == 33


def test_one_round_grid_deals_compact_blocks():
    # 4096x4096 at 256^2 tiles (16 x 16 tiles, one round of 8 x 32 workers): an
    # 8-row band holds 128 tiles, fewer than the 256 workers, so every XCD gets
    # one whole 8 x 4 block (12 panels) instead of two 8 x 2 strips (18)
    order, off, quota = asym.schedule_build(16, 16, [32] * 8, asym.MAP_AWARE)
    assert quota == [32] * 8
    blocks = set()
    for x in range(8):
        mine = order[off[x]:off[x + 1]]
        rows = {t // 16 for t in mine}
        cols = {t % 16 for t in mine}
        assert len(rows) == 8 and len(cols) == 4 and max(cols) - min(cols) == 3
        blocks.add((min(rows), min(cols)))
    assert blocks == {(r, c) for r in (0, 8) for c in (0, 4, 8, 12)}
    # block k (band by band, left to right) on XCD k mod 8
    assert [min(order[off[x]:off[x + 1]]) for x in range(8)] == [0, 4, 8, 12, 128, 132, 136, 140]
    # the band runs stay where a band holds a whole round (8192^3) or the
    # counts are unequal
    assert osched.block_deal_lists(32, 32, [32] * 8, 8) is None
    assert osched.block_deal_lists(16, 16, [16, 10, 22, 16, 13, 19, 16, 16], 4) is None
    # an explicit band keeps the band runs
    order_b, _, _ = asym.schedule_build(16, 16, [32] * 8, asym.MAP_AWARE, band=8)
    assert order_b == [t for lst in osched.aware_lists(16, 16, [32] * 8, 8) for t in lst]


@pytest.mark.parametrize("args", [
    (0, 4, [1] * 8, 0), (4, 4, [0] * 8, 0), (4, 4, [1] * 8, 7), (4, 4, [-1] + [1] * 7, 0)])
def test_schedule_rejects_bad_input(lib, args):
    with pytest.raises(asym.AsymError) as e:
        asym.schedule_build(*args)
    assert e.value.status == asym.EINVAL


# -- topology from synthetic records ------------------------------------------------

def fake_records(layout, n_rep=4, seed=0, rr=True):
    """layout: {xcc: [(se, sh, cu), ...]} -> identity records, shuffled."""
    rng = random.Random(seed)
    cus = [(x, se, sh, cu) for x, lst in layout.items() for (se, sh, cu) in lst]
    recs = []
    nx = max(layout) + 1
    for rep in range(n_rep):
        for c in rng.sample(cus, len(cus)):
            b = len(recs)
            x = c[0]
            if rr:
                # place the record at a block index whose residue is its XCC
                b = b - (b % nx) + x
            hw = (c[3] << 8) | (c[2] << 12) | (c[1] << 13) | (rng.randint(0, 15))
            recs.append([x | (rng.randint(0, 15) << 8), hw, b, 0])
    return recs


def uniform_layout(n_xcc=8, n_se=4, per_se=8):
    return {x: [(se, 0, cu) for se in range(n_se) for cu in range(per_se)] for x in range(n_xcc)}


def test_topology_uniform_matches_oracle(lib):
    lay = uniform_layout()
    recs = fake_records(lay)
    t = asym.topology_from_records(recs, 256, 8)
    info = t.info()
    assert info["n_cus"] == 256 and info["cus_per_xcd"] == [32] * 8
    cus = [(c["xcc"], c["se"], c["sh"], c["cu"]) for c in t.cus()]
    assert cus == otopo.build_map(recs)
    assert otopo.invariant_violations(cus, 256, 8) == []
    assert t.dispatch_rr_fraction() == pytest.approx(otopo.round_robin_fraction(recs, 8))
    js = t.json()
    assert js["n_cus"] == 256 and len(js["cus"]) == 256


def test_topology_uneven_floorswept_layout(lib):
    # floorsweeping leaves XCDs (and SEs) with different CU counts
    rng = random.Random(7)
    lay = {}
    for x in range(8):
        lst = [(se, sh, cu) for se in range(4) for sh in range(2) for cu in range(5)]
        lay[x] = sorted(rng.sample(lst, rng.randint(20, 36)))
    n = sum(len(v) for v in lay.values())
    recs = fake_records(lay, seed=3)
    t = asym.topology_from_records(recs, n, 8)
    cus = [(c["xcc"], c["se"], c["sh"], c["cu"]) for c in t.cus()]
    assert cus == otopo.build_map(recs)
    assert t.info()["cus_per_xcd"] == otopo.per_xcd_counts(cus, 8)


def test_topology_rejects_broken_maps(lib):
    lay = uniform_layout()
    recs = fake_records(lay)
    # the device reports a different CU count than the records show
    with pytest.raises(asym.AsymError) as e:
        asym.topology_from_records(recs, 250, 8)
    assert e.value.status == asym.EINVARIANT
    # an XCD missing entirely
    lay7 = {x: v for x, v in lay.items() if x != 5}
    recs7 = fake_records(lay7)
    with pytest.raises(asym.AsymError) as e:
        asym.topology_from_records(recs7, 224, 8)
    assert e.value.status == asym.EINVARIANT
    assert otopo.invariant_violations(otopo.build_map(recs7), 224, 8) != []
    # XCC id beyond the device's XCC count
    with pytest.raises(asym.AsymError) as e:
        asym.topology_from_records(recs, 256, 4)
    assert e.value.status == asym.EINVARIANT
    # a mask-bit map that sends two bits to one CU
    bit_rec = list(range(256))
    first = {}
    for i, r in enumerate(recs):
        first.setdefault(otopo.fields(r[0], r[1]), i)
    keys = otopo.build_map(recs)
    bit_rec = [first[keys[b]] for b in range(256)]
    bad = list(bit_rec)
    bad[1] = bad[0]
    with pytest.raises(asym.AsymError) as e:
        asym.topology_from_records(recs, 256, 8, bad)
    assert e.value.status == asym.EINVARIANT


def _maskmap_topology(seed=0):
    lay = uniform_layout()
    recs = fake_records(lay, seed=seed)
    first = {}
    for i, r in enumerate(recs):
        first.setdefault(otopo.fields(r[0], r[1]), i)
    keys = otopo.build_map(recs)
    # bit b -> CU on XCC b % 8 (interleaved), a permutation of the dense order
    perm = []
    per_x = {x: [k for k in keys if k[0] == x] for x in range(8)}
    for b in range(256):
        perm.append(per_x[b % 8][b // 8])
    bit_rec = [first[k] for k in perm]
    return asym.topology_from_records(recs, 256, 8, bit_rec), perm


def test_maskmap_and_cusets(lib):
    t, perm = _maskmap_topology()
    cus = t.cus()
    assert sorted(c["mask_bit"] for c in cus) == list(range(256))
    for c in cus:
        assert perm[c["mask_bit"]] == (c["xcc"], c["se"], c["sh"], c["cu"])
    # XCD-aligned: whole XCDs
    m = t.cuset(64, asym.CUSET_XCD_ALIGNED)
    assert len(m) == 64 and t.cuset_counts(m) == [32, 32, 0, 0, 0, 0, 0, 0]
    m2 = t.cuset(64, asym.CUSET_XCD_ALIGNED, exclude=m)
    assert not set(m) & set(m2) and t.cuset_counts(m2) == [0, 0, 32, 32, 0, 0, 0, 0]
    with pytest.raises(asym.AsymError):
        t.cuset(48, asym.CUSET_XCD_ALIGNED)
    # striped: the same share of every XCD, balanced over shader engines
    s = t.cuset(64, asym.CUSET_STRIPED)
    assert t.cuset_counts(s) == [8] * 8
    by_se = {}
    for b in s:
        x, se, _, _ = perm[b]
        by_se[(x, se)] = by_se.get((x, se), 0) + 1
    assert set(by_se.values()) == {2}
    rest = t.cuset(192, asym.CUSET_STRIPED, exclude=s)
    assert sorted(s + rest) == list(range(256))
    # random: seeded, reproducible, honours exclusion
    r1 = t.cuset(128, asym.CUSET_RANDOM, seed=4)
    r2 = t.cuset(128, asym.CUSET_RANDOM, seed=4)
    r3 = t.cuset(128, asym.CUSET_RANDOM, seed=5)
    assert r1 == r2 and r1 != r3 and len(r1) == 128
    r4 = t.cuset(100, asym.CUSET_RANDOM, seed=1, exclude=r1)
    assert not set(r4) & set(r1)


def test_xcd_split_lends_one_cu_per_foreign_xcd(lib):
    t, perm = _maskmap_topology()
    a, b = t.cuset_split_xcds(0x0F)
    assert not set(a) & set(b) and sorted(a + b) == list(range(256))
    assert t.cuset_counts(a) == [31, 31, 31, 31, 1, 1, 1, 1]
    assert t.cuset_counts(b) == [1, 1, 1, 1, 31, 31, 31, 31]
    # the lent CU is the lowest CU of its XCD in the dense order
    lowest = {}
    for c in t.cus():
        lowest.setdefault(c["xcc"], c["mask_bit"])
    for x in range(8):
        owner, other = (a, b) if x < 4 else (b, a)
        assert lowest[x] in other and lowest[x] not in owner
    a6, b2 = t.cuset_split_xcds(0x3F)
    assert t.cuset_counts(a6) == [31] * 6 + [1, 1] and t.cuset_counts(b2) == [1] * 6 + [31, 31]
    for bad in (0, 0xFF, 0x100):
        with pytest.raises(asym.AsymError):
            t.cuset_split_xcds(bad)
    plain = asym.topology_from_records(fake_records(uniform_layout()), 256, 8)
    with pytest.raises(asym.AsymError) as e:
        plain.cuset_split_xcds(0x0F)
    assert e.value.status == asym.EUNSUPPORTED


def test_masked_stream_refuses_an_empty_xcd(lib):
    t, _ = _maskmap_topology()
    aligned = t.cuset(128, asym.CUSET_XCD_ALIGNED)
    with pytest.raises(asym.AsymError) as e:
        asym.stream_create(t, aligned)
    assert e.value.status == asym.EUNSUPPORTED
    # a partial mask needs a mask map
    plain = asym.topology_from_records(fake_records(uniform_layout()), 256, 8)
    with pytest.raises(asym.AsymError) as e:
        plain.cuset_counts(list(range(100)))
    assert e.value.status == asym.EUNSUPPORTED


def test_gemm_and_copy_argument_errors(lib):
    vp = 0x1000
    lib_ = asym.load_library()
    import ctypes
    P = ctypes.c_void_p(vp)
    cases = [
        ((None, 0, 4, 4, P, 4, P, 4, 0, P, 4, 0, 0, None), asym.EINVAL),      # M = 0
        ((None, 4, 4, 4, None, 4, P, 4, 0, P, 4, 0, 0, None), asym.EINVAL),   # null A
        ((None, 4, 4, 8, P, 4, P, 8, 0, P, 4, 0, 0, None), asym.EINVAL),      # lda < K
        ((None, 4, 8, 4, P, 4, P, 4, 1, P, 8, 0, 0, None), asym.EINVAL),      # [K][N] B, ldb < N
        ((None, 4, 4, 4, P, 4, P, 4, 7, P, 4, 0, 0, None), asym.EINVAL),      # bad layout
        ((None, 4, 4, 4, P, 4, P, 4, 0, P, 4, 9, 0, None), asym.EINVAL),      # bad mapping
    ]
    for args, want in cases:
        assert lib_.asym_gemm_bf16(*args) == want, args
        assert asym.last_error()
    Q = ctypes.c_void_p(vp + 4096)
    assert lib_.asym_copy_bf16(None, Q, P, 24, 1, None, 0, None) == asym.EINVAL     # size not 16k
    assert lib_.asym_copy_bf16(None, Q, P, 32, 0, None, 0, None) == asym.EINVAL     # no pass
    assert lib_.asym_copy_bf16(None, P, P, 32, 1, None, 0, None) == asym.EINVAL     # overlap
    assert lib_.asym_copy_bf16(None, ctypes.c_void_p(vp + 8), P, 32, 1, None, 0, None) == asym.EINVAL


def _grouped_cases():
    rng = random.Random(99)
    cases = [([1] * 32, 16, [32] * 8), ([5, 4, 4, 5, 4, 5], 16, [32] * 8), ([0, 3, 0, 1], 7, [32] * 8),
             ([2, 1], 28, [16, 10, 22, 16, 13, 19, 16, 16]), ([4], 1, [1, 0, 0, 0, 0, 0, 0, 0])]
    for _ in range(20):
        G = rng.randint(1, 12)
        n = rng.choice([1, 2, 4, 8])
        slots = [rng.randint(0, 32) for _ in range(n)]
        if sum(slots) == 0:
            slots[0] = 1
        cases.append(([rng.randint(0, 6) for _ in range(G)], rng.randint(1, 30), slots))
    return cases


@pytest.mark.parametrize("rows,tn,slots", _grouped_cases())
def test_grouped_schedule_matches_oracle(lib, rows, tn, slots):
    T = sum(rows) * tn
    order, off, quota = asym.grouped_schedule_build(rows, tn, slots, asym.MAP_AWARE)
    lists = osched.grouped_aware_lists(rows, tn, slots)
    assert quota == [len(lst) for lst in lists]
    assert order == [t for lst in lists for t in lst]
    assert off[0] == 0 and all(off[x + 1] - off[x] == quota[x] for x in range(len(slots)))
    assert sorted(order) == list(range(T))                     # every tile exactly once
    W = sum(slots)
    n_groups = sum(1 for r in rows if r)
    assert all(abs(quota[x] - T * slots[x] / W) < max(1, n_groups) for x in range(len(slots)))
    assert all(q == 0 for q, s in zip(quota, slots) if s == 0)
    order_g, _, quota_g = asym.grouped_schedule_build(rows, tn, slots, asym.MAP_OBLIVIOUS_GROUPED)
    assert order_g == osched.grouped_oblivious_order(rows, tn, True)
    owner = osched.oblivious_assignment(order_g, slots)
    assert quota_g == [sum(1 for v in owner.values() if v == x) for x in range(len(slots))]
    order_r, _, _ = asym.grouped_schedule_build(rows, tn, slots, asym.MAP_OBLIVIOUS_ROWMAJOR)
    assert order_r == osched.grouped_oblivious_order(rows, tn, False)


def test_grouped_aware_keeps_a_column_panel_on_one_xcd():
    """Six groups of 4-5 tile rows on 8 XCDs of 32: every column panel of a
    group (its tile rows of one column) lands on at most two XCDs."""
    rows, tn, slots = [5, 4, 4, 4, 4, 5], 16, [32] * 8
    order, off, _ = asym.grouped_schedule_build(rows, tn, slots, asym.MAP_AWARE)
    owner = {t: x for x in range(8) for t in order[off[x]:off[x + 1]]}
    ids = osched.grouped_tile_ids(rows, tn)
    for g, r_g in enumerate(rows):
        for c in range(tn):
            assert len({owner[ids[(g, r, c)]] for r in range(r_g)}) <= 2


def test_grouped_schedule_rejects_bad_input(lib):
    with pytest.raises(asym.AsymError):
        asym.grouped_schedule_build([], 4, [32] * 8, asym.MAP_AWARE)
    with pytest.raises(asym.AsymError):
        asym.grouped_schedule_build([1, -1], 4, [32] * 8, asym.MAP_AWARE)
    with pytest.raises(asym.AsymError):
        asym.grouped_schedule_build([1, 1], 0, [32] * 8, asym.MAP_AWARE)
    with pytest.raises(asym.AsymError):
        asym.grouped_schedule_build([1, 1], 4, [0] * 8, asym.MAP_AWARE)


def test_dispatch_share_counts_classes_not_the_start():
    """The dispatch share is per residue class of block indices: dealing that
    starts on another XCD (a rotation) still puts each class on one XCD and
    scores 1; a class split over two XCDs scores the larger half.  Oracle and
    library agree on both."""
    lay = uniform_layout()
    recs = fake_records(lay)
    rotated = [[((r[0] & 0xF) + 3) % 8 | (r[0] & ~0xF), r[1], r[2], r[3]] for r in recs]
    assert otopo.round_robin_fraction(rotated, 8) == 1.0
    # the XCC field no longer matches the layout's CU records, so only the share is compared
    split = [list(r) for r in recs]
    cls0 = [r for r in split if r[2] % 8 == 0]
    for r in cls0[: len(cls0) // 4]:
        r[0] = (r[0] & ~0xF) | 1          # a quarter of class 0 moved to XCC 1
    want = 1.0 - (len(cls0) // 4) / len(split)
    assert abs(otopo.round_robin_fraction(split, 8) - want) < 1e-12


# -- per-chip topology cache ------------------------------------------------------------

def test_topology_cache_round_trip_and_staleness(lib, tmp_path):
    """A saved map loads back equal under its key, is refused under another key
    (another chip or partition mode), when it lacks a requested probe, and
    when the file is missing, truncated or edited to break an invariant."""
    t, perm = _maskmap_topology(seed=5)
    key = "pci=0000:0a:00.0 uuid=00ff hip=70200000 driver=70200000 arch=gfx950 compute=SPX memory=NPS1 cus=256 xccs=8"
    path = str(tmp_path / "topo.txt")
    t.save(path, key)
    u = asym.topology_load(path, key, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP)
    ju, jt = u.json(), t.json()
    assert ju["cus"] == jt["cus"] and ju["cus_per_xcd"] == jt["cus_per_xcd"] and ju["has_maskmap"]
    assert ju["key"] == key and jt["key"] == "records"
    assert [u.cu(i)["mask_bit"] for i in range(256)] == [t.cu(i)["mask_bit"] for i in range(256)]
    assert u.cuset_counts(list(range(0, 256, 2))) == t.cuset_counts(list(range(0, 256, 2)))
    # another chip, another partition mode
    for other in (key.replace("0a:00.0", "0b:00.0"), key.replace("compute=SPX", "compute=CPX"),
                  key.replace("memory=NPS1", "memory=NPS2")):
        with pytest.raises(asym.AsymError) as e:
            asym.topology_load(path, other, asym.PROBE_IDENTITY)
        assert e.value.status == asym.ENOCACHE and "another key" in str(e.value)
    # a probe the cached map does not hold
    with pytest.raises(asym.AsymError) as e:
        asym.topology_load(path, key, asym.PROBE_IDENTITY | asym.PROBE_LATENCY)
    assert e.value.status == asym.ENOCACHE and "lacks" in str(e.value)
    # missing file
    with pytest.raises(asym.AsymError) as e:
        asym.topology_load(str(tmp_path / "none.txt"), key)
    assert e.value.status == asym.ENOCACHE
    lines = open(path).read().splitlines()
    # truncated
    open(path, "w").write("\n".join(lines[:100]) + "\n")
    with pytest.raises(asym.AsymError) as e:
        asym.topology_load(path, key)
    assert e.value.status == asym.ENOCACHE
    # two CU lines made equal: the exact invariants reject the map
    cu_lines = [i for i, l in enumerate(lines) if l.startswith("cu ")]
    bad = list(lines)
    f0 = bad[cu_lines[0]].split()
    f1 = bad[cu_lines[1]].split()
    bad[cu_lines[1]] = " ".join(f0[:5] + f1[5:])
    open(path, "w").write("\n".join(bad) + "\n")
    with pytest.raises(asym.AsymError) as e:
        asym.topology_load(path, key)
    assert e.value.status == asym.ENOCACHE and "invariant" in str(e.value)
    # a mask bit used twice
    bad = list(lines)
    f1 = bad[cu_lines[1]].split()
    bad[cu_lines[1]] = " ".join(f1[:5] + [bad[cu_lines[0]].split()[5]])
    open(path, "w").write("\n".join(bad) + "\n")
    with pytest.raises(asym.AsymError) as e:
        asym.topology_load(path, key, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP)
    assert e.value.status == asym.ENOCACHE
    # identity-only map: loads for identity requests only
    plain = asym.topology_from_records(fake_records(uniform_layout()), 256, 8)
    plain.save(path, key)
    assert asym.topology_load(path, key).info()["cus_per_xcd"] == [32] * 8
    with pytest.raises(asym.AsymError):
        asym.topology_load(path, key, asym.PROBE_MASKMAP)


def test_noalloc_rejections_need_no_device(lib):
    """The no-allocation GEMM refuses, before any device call, what its fixed
    per-GPU array cannot serve: no topology (a first-use probe would
    allocate), B stored [K][N] (a transposed copy would be needed), and more
    output tiles than the array's schedule holds."""
    import ctypes
    lib_ = asym.load_library()
    lim = asym.noalloc_limits()
    assert lim["scratch_bytes"] == (17 << 20) and lim["max_tiles"] == ((1 << 20) - 512) // 4
    assert lim["max_partial_bytes"] == 16 << 20
    t = asym.topology_from_records(fake_records(uniform_layout()), 256, 8)
    P = ctypes.c_void_p(0x1000)
    assert lib_.asym_gemm_bf16_noalloc(None, 64, 64, 64, P, 64, P, 64, 0, P, 64, 0, 0, None) == asym.EINVAL
    assert "topology" in asym.last_error()
    assert lib_.asym_gemm_bf16_noalloc(t.handle, 64, 64, 64, P, 64, P, 64, 1, P, 64, 0, 0, None) == \
        asym.EUNSUPPORTED
    side = 131072  # 512 x 512 tiles of 256 > 262016
    assert lib_.asym_gemm_bf16_noalloc(t.handle, side, side, 8, P, 8, P, 8, 0, P, side, 0, 0, None) == \
        asym.EINVAL
    assert "output tiles" in asym.last_error()


def test_mla_form_level_switch(lib):
    """The latent-attention kernel-form level round-trips (0 wave form only,
    1 up to the 64-head form, 2 the default, 3 the 128-head form wherever it
    fits) and other levels are refused without changing it."""
    prev = asym.set_mla_workgroup_form(1)
    try:
        assert prev == 2
        assert asym.set_mla_workgroup_form(False) == 1
        assert asym.set_mla_workgroup_form(True) == 0
        assert asym.set_mla_workgroup_form(3) == 2
        assert lib.asym_mla_set_workgroup_form(4) == asym.EINVAL
        assert lib.asym_mla_set_workgroup_form(-1) == asym.EINVAL
        with pytest.raises(asym.AsymError):
            asym.set_mla_workgroup_form(7)
        assert asym.set_mla_workgroup_form(2) == 3
    finally:
        asym.set_mla_workgroup_form(prev)
