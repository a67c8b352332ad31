"""Home map and local / remote chunk lists: pins for the oracle, then the
library's host code against the oracle (no GPU).

The oracle's chunk homes are pinned to the planted truth of a synthetic region
(one parity over the address bits, a random bit per 2 MiB page): every chunk's
home must equal the planted home of its first byte, and so must the
verification lines.  The lists are pinned by their invariants: every chunk at
most once, each XCD reading only chunks homed on its own group (LOCAL) or on
the other one (REMOTE), round-robin balance, nothing for inactive XCDs.
"""
import numpy as np
import pytest

import paper_2609_24270_amd as asym
from oracle import numa as onuma
from paper_2609_24270_amd import workloads

GRP = [0, 0, 0, 0, 1, 1, 1, 1]
MI355X_LIKE = (1 << 13) | (1 << 21) | (1 << 28)


def _oracle_map(seed, n_pages, mask, chunk_log2, n_verify=64):
    Lp, vo, Lv, home_of = workloads.planted_home_region(seed, n_pages, mask, n_verify)
    pages = onuma.homes_given_groups(Lp.tolist(), GRP, 20.0)
    chunks = onuma.chunk_homes(pages, mask, chunk_log2)
    vh = onuma.homes_given_groups(Lv.tolist(), GRP, 20.0)
    return Lp, vo, Lv, home_of, pages, chunks, vh


@pytest.mark.parametrize("mask,chunk_log2", [(MI355X_LIKE, 13), (MI355X_LIKE, 12),
                                             ((1 << 14) | (1 << 17) | (1 << 22), 14),
                                             (1 << 25, 21)])
def test_oracle_chunk_homes_equal_the_planted_homes(mask, chunk_log2):
    Lp, vo, Lv, home_of, pages, chunks, vh = _oracle_map(3, 24, mask, chunk_log2)
    assert len(chunks) == (24 << 21) >> chunk_log2
    assert chunks == [home_of(c << chunk_log2) for c in range(len(chunks))]
    # a chunk is one home: its last line agrees with its first
    assert chunks == [home_of(((c + 1) << chunk_log2) - 128) for c in range(len(chunks))]
    assert vh == [home_of(o) for o in vo]
    assert vh == [chunks[o >> chunk_log2] for o in vo]


def test_oracle_rejects_a_hash_below_the_chunk():
    with pytest.raises(ValueError):
        onuma.chunk_homes([0, 1], MI355X_LIKE, 14)


def test_oracle_homes_tie_and_pairs():
    # within a 2 MiB page chunk pairs (2j, 2j+1) of 8 KiB differ only in bit 13,
    # so each pair holds one chunk of each home
    _, _, _, _, pages, chunks, _ = _oracle_map(4, 8, MI355X_LIKE, 13)
    assert all(chunks[2 * j] != chunks[2 * j + 1] for j in range(len(chunks) // 2))
    lat = [[800] * 3 for _ in range(4)] + [[812] * 3 for _ in range(4)]
    assert onuma.homes_given_groups(lat, GRP, 20.0) == [-1, -1, -1]
    assert onuma.homes_given_groups(lat, GRP, 12.0) == [0, 0, 0]
    assert onuma.chunk_homes([-1, 1], 1 << 13, 13)[:2] == [-1, -1]


@pytest.mark.parametrize("mode", [onuma.ALL, onuma.LOCAL, onuma.REMOTE])
@pytest.mark.parametrize("xcd_mask", [0, 0x0F, 0x33, 0x80])
def test_oracle_lists_invariants(mode, xcd_mask):
    g = np.random.default_rng(5)
    home = [int(v) for v in g.choice([-1, 0, 1], size=1000, p=[0.05, 0.5, 0.45])]
    out, off = onuma.chunk_lists(home, 8, GRP, xcd_mask, mode)
    active = [x for x in range(8) if xcd_mask == 0 or (xcd_mask >> x) & 1]
    assert off[0] == 0 and off[-1] == len(out) and all(a <= b for a, b in zip(off, off[1:]))
    assert len(set(out)) == len(out)
    per = {x: out[off[x]:off[x + 1]] for x in range(8)}
    assert all(not per[x] for x in range(8) if x not in active)
    if mode == onuma.ALL:
        assert sorted(out) == list(range(1000))
        sizes = [len(per[x]) for x in active]
        assert max(sizes) - min(sizes) <= 1
    else:
        for x in active:
            want = GRP[x] if mode == onuma.LOCAL else 1 - GRP[x]
            assert all(home[c] == want for c in per[x])
        readable = {h for h in (0, 1)
                    if any((GRP[x] if mode == onuma.LOCAL else 1 - GRP[x]) == h for x in active)}
        assert sorted(out) == [c for c in range(1000) if home[c] in readable]
        for h in readable:
            xs = [x for x in active if (GRP[x] if mode == onuma.LOCAL else 1 - GRP[x]) == h]
            sizes = [len(per[x]) for x in xs]
            assert max(sizes) - min(sizes) <= 1


@pytest.mark.parametrize("mask,chunk_log2,n_pages", [(MI355X_LIKE, 13, 24), ((1 << 14) | (1 << 23), 14, 9),
                                                     (1 << 13, 13, 1)])
def test_library_home_map_analysis_matches_oracle(mask, chunk_log2, n_pages):
    Lp, vo, Lv, home_of, pages, chunks, vh = _oracle_map(6, n_pages, mask, chunk_log2, n_verify=100)
    L = np.concatenate([Lp, Lv], axis=1)
    info, homes = asym.home_map_analyze(L, n_pages, vo, GRP, mask, chunk_log2)
    assert homes.tolist() == chunks
    assert info["n_pages"] == n_pages and info["n_chunks"] == len(chunks)
    assert info["unclassified_pages"] == pages.count(-1)
    assert info["chunk_share"][0] == chunks.count(0) / len(chunks)
    assert info["verify_classified"] == sum(1 for h in vh if h >= 0) == 100
    assert info["verify_agree"] == 100
    loc = [Lp[x][p] for x in range(8) for p in range(n_pages) if pages[p] >= 0 and pages[p] == GRP[x]]
    rem = [Lp[x][p] for x in range(8) for p in range(n_pages) if pages[p] >= 0 and pages[p] != GRP[x]]
    assert abs(info["local_cycles"] - (sum(loc) / len(loc) if loc else -1.0)) < 1e-9
    assert abs(info["remote_cycles"] - (sum(rem) / len(rem) if rem else -1.0)) < 1e-9


def test_library_home_map_analysis_counts_disagreement():
    """A verification line whose measured home contradicts the map is counted
    as a disagreement (the planted latencies of one line are swapped)."""
    Lp, vo, Lv, home_of, pages, chunks, vh = _oracle_map(7, 16, MI355X_LIKE, 13, n_verify=10)
    Lv = Lv.copy()
    Lv[:, 3] = np.concatenate([Lv[4:, 3], Lv[:4, 3]])
    info, _ = asym.home_map_analyze(np.concatenate([Lp, Lv], axis=1), 16, vo, GRP, MI355X_LIKE, 13)
    assert info["verify_classified"] == 10 and info["verify_agree"] == 9


@pytest.mark.parametrize("mode", [asym.CHUNKS_ALL, asym.CHUNKS_LOCAL, asym.CHUNKS_REMOTE])
@pytest.mark.parametrize("xcd_mask", [0, 0x0F, 0x33, 0x80])
def test_library_lists_match_oracle(mode, xcd_mask):
    g = np.random.default_rng(8)
    home = g.choice([-1, 0, 1], size=777, p=[0.05, 0.5, 0.45]).astype(np.int8)
    out, off = asym.chunk_lists(home, 8, GRP, mode, xcd_mask)
    ref_out, ref_off = onuma.chunk_lists([int(v) for v in home], 8, GRP, xcd_mask, mode)
    assert out.tolist() == ref_out and off.tolist() == ref_off


def test_library_rejects_bad_input():
    Lp, vo, Lv, *_ = _oracle_map(9, 4, MI355X_LIKE, 13, n_verify=2)
    L = np.concatenate([Lp, Lv], axis=1)
    for kw in (dict(chunk_log2=14), dict(chunk_log2=11), dict(chunk_log2=22)):
        with pytest.raises(asym.AsymError):
            asym.home_map_analyze(L, 4, vo, GRP, MI355X_LIKE, **kw)
    with pytest.raises(asym.AsymError):
        asym.home_map_analyze(L, 4, vo, [0, 0, 0, 0, 1, 1, 1, 2], MI355X_LIKE, 13)
    with pytest.raises(asym.AsymError):
        asym.home_map_analyze(L, 4, vo, [0] * 8, MI355X_LIKE, 13)
    with pytest.raises(asym.AsymError):
        asym.home_map_analyze(L, 4, [0, 5 << 21], GRP, MI355X_LIKE, 13)   # line beyond the range
    home = np.zeros(10, dtype=np.int8)
    with pytest.raises(asym.AsymError):
        asym.chunk_lists(home, 8, GRP, 3)
    with pytest.raises(asym.AsymError):
        asym.chunk_lists(home, 8, GRP, asym.CHUNKS_LOCAL, xcd_mask=0x100)
    with pytest.raises(asym.AsymError):
        asym.chunk_lists(home, 8, None, asym.CHUNKS_LOCAL)
