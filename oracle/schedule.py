"""Oracle for the tile schedule.  TEST INFRASTRUCTURE ONLY.

Section 7.1 assigns each persistent block the tasks local to its partition and
spreads the work over partitions in proportion to their compute units; the
full-GPU lesson of Section 7.4 restates the proportional rule.  "In proportion"
with whole tiles is an apportionment problem; the reading taken here is
Hamilton's largest-remainder method (each partition first gets the floor of its
exact share T*w_x/W, and the tiles left over go one each to the largest
fractional remainders, ties to the lower partition index).

The tile order is the banded column-major walk: tile rows are cut into bands of
`band` rows, each band is walked column by column, top to bottom.  AWARE shares
every band out among the partitions: the band's walk is cut into contiguous
runs of Hamilton-apportioned lengths, one per partition in index order, and a
partition's list is its run of band 0, then of band 1, and so on.  A second
reading of "tasks local to the partition" covers grids whose band holds fewer
tiles than one round of every partition's workers (band * tiles_n < n * s): a
band's runs would then be strips band rows by a few columns, taken from two or
more bands at once.  With s workers on every partition the grid is instead cut
into band x (s / band) blocks, numbered band by band and left to right, and
block k goes to partition k mod n (each block's tiles column by column, top to
bottom), where the blocks divide the grid and come out even.  The
oblivious mappings hand order position i of the whole walk to workgroup
i mod P, which round-robin dispatch places on partition (i mod P) mod n.

Written from the definitions with exact rational arithmetic; no code is shared
with the library.
"""
from __future__ import annotations

from fractions import Fraction


def hamilton_quotas(total: int, weights):
    W = sum(weights)
    if W <= 0 or total <= 0:
        return [0] * len(weights)
    shares = [Fraction(total * w, W) for w in weights]
    q = [int(s) for s in shares]            # floor (shares are >= 0)
    left = total - sum(q)
    rema = [(s - int(s), -i) for i, s in enumerate(shares)]
    ranked = sorted(range(len(weights)), key=lambda i: rema[i], reverse=True)
    for i in ranked:
        if left == 0:
            break
        if weights[i] > 0:
            q[i] += 1
            left -= 1
    return q


def banded_order(tiles_m: int, tiles_n: int, band: int):
    order = []
    r0 = 0
    while r0 < tiles_m:
        rows = range(r0, min(tiles_m, r0 + band))
        for c in range(tiles_n):
            for r in rows:
                order.append(r * tiles_n + c)
        r0 += band
    return order


def rowmajor_order(tiles_m: int, tiles_n: int):
    return list(range(tiles_m * tiles_n))


def band_walks(tiles_m: int, tiles_n: int, band: int):
    """The banded walk, one list per band."""
    walks = []
    r0 = 0
    while r0 < tiles_m:
        rows = range(r0, min(tiles_m, r0 + band))
        walks.append([r * tiles_n + c for c in range(tiles_n) for r in rows])
        r0 += band
    return walks


def aware_lists(tiles_m, tiles_n, slots, band):
    """Per-partition tile lists of the aware mapping."""
    lists = [[] for _ in slots]
    for walk in band_walks(tiles_m, tiles_n, band):
        q = hamilton_quotas(len(walk), slots)
        pos = 0
        for x, qx in enumerate(q):
            lists[x].extend(walk[pos:pos + qx])
            pos += qx
    return lists


def block_deal_lists(tiles_m, tiles_n, slots, band):
    """The block-dealing form of the aware lists (module docstring), or None
    where it does not apply: unequal worker counts, a band that already holds
    a round of every partition, or blocks that do not divide the grid or do
    not come out even over the partitions."""
    n = len(slots)
    s = slots[0]
    if s < 1 or any(w != s for w in slots):
        return None
    h = band
    if h < 1 or s % h or tiles_m % h:
        return None
    c = s // h
    if tiles_n % c or h * tiles_n >= n * s:
        return None
    if (tiles_m * tiles_n // s) % n:
        return None
    lists = [[] for _ in slots]
    k = 0
    for r0 in range(0, tiles_m, h):
        for c0 in range(0, tiles_n, c):
            lists[k % n].extend(r * tiles_n + cc for cc in range(c0, c0 + c) for r in range(r0, r0 + h))
            k += 1
    return lists


def aware_lists_auto(tiles_m, tiles_n, slots):
    """The aware lists with the band chosen by band_cost_choice: dealt blocks
    where they apply, else the band runs."""
    band = band_cost_choice(tiles_m, max(slots))
    lists = block_deal_lists(tiles_m, tiles_n, slots, band)
    return lists if lists is not None else aware_lists(tiles_m, tiles_n, slots, band)


def aware_assignment(tiles_m, tiles_n, slots, band):
    """tile id -> partition, and the per-partition tile counts."""
    lists = aware_lists(tiles_m, tiles_n, slots, band)
    owner = {t: x for x, lst in enumerate(lists) for t in lst}
    return owner, [len(lst) for lst in lists]


def oblivious_assignment(order, slots):
    """tile id -> partition under round-robin dispatch of workgroup i mod P."""
    P = sum(slots)
    n = len(slots)
    return {t: (i % P) % n for i, t in enumerate(order)}


def band_cost_choice(tiles_m: int, s: int) -> int:
    """Band height minimising band + ceil(s/band); ties to a band dividing
    tiles_m, then to the taller band."""
    s = max(1, s)
    best = None
    for h in range(1, min(tiles_m, s) + 1):
        key = (h + -(-s // h), 0 if tiles_m % h == 0 else 1, -h)
        if best is None or key < best[0]:
            best = (key, h)
    return best[1]


# ---- grouped GEMM -------------------------------------------------------------
# The same recipe applied to grouped GEMM (Section 7.1: the expert layer of
# mixture-of-experts models).  Group g owns rows_g tile rows of tiles_n
# columns.  A tile is named (g, r, c); the tiles are numbered group after
# group, row-major inside a group.  Reading taken here: each group is one band
# of the plain schedule, so the aware mapping shares every group out among the
# partitions exactly as it shares out a band.

def grouped_tile_ids(rows_per_group, tiles_n):
    """(g, r, c) -> tile id, numbering groups in order, row-major inside each."""
    ids, nxt = {}, 0
    for g, rows in enumerate(rows_per_group):
        for r in range(rows):
            for c in range(tiles_n):
                ids[(g, r, c)] = nxt
                nxt += 1
    return ids


def grouped_walks(rows_per_group, tiles_n):
    """One walk per group: column by column, each column top to bottom."""
    ids = grouped_tile_ids(rows_per_group, tiles_n)
    return [[ids[(g, r, c)] for c in range(tiles_n) for r in range(rows)]
            for g, rows in enumerate(rows_per_group)]


def grouped_aware_lists(rows_per_group, tiles_n, slots):
    lists = [[] for _ in slots]
    for walk in grouped_walks(rows_per_group, tiles_n):
        if not walk:
            continue
        q = hamilton_quotas(len(walk), slots)
        pos = 0
        for x, qx in enumerate(q):
            lists[x].extend(walk[pos:pos + qx])
            pos += qx
    return lists


def grouped_oblivious_order(rows_per_group, tiles_n, grouped_walk: bool):
    if grouped_walk:
        return [t for walk in grouped_walks(rows_per_group, tiles_n) for t in walk]
    return list(range(sum(rows_per_group) * tiles_n))
