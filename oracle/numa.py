"""Oracle for the home map of an allocation and the chunk lists of the
local / remote read study.  TEST INFRASTRUCTURE ONLY.

Section 6.1 classifies every page of a contiguous region by its partition and
then reads only local or only remote pages; the appendix on NUMA-aware address
remapping places data by the same classification.  Readings taken here:
  * an address's partition is its home group: with two XCD groups, the group
    whose XCDs see the lower mean latency, none when the two means differ by
    less than a tie margin;
  * the home of a chunk is the home of its 2 MiB page's first line XOR the
    parity of (the chunk's offset inside the page AND the partition hash),
    which is what one parity over the address bits gives when the page's
    higher bits are fixed; a page with no home gives its chunks none;
  * the read lists: ALL deals every chunk round-robin over the active XCDs in
    chunk order; LOCAL deals each group's chunks round-robin over that group's
    active XCDs; REMOTE over the other group's active XCDs; chunks with no home
    or no reader are left out.
Plain Python; no code shared with the library.
"""
from __future__ import annotations

PAGE = 2 << 20
ALL, LOCAL, REMOTE = 0, 1, 2


def parity(v: int) -> int:
    return bin(v).count("1") & 1


def homes_given_groups(lat, grp, tie: float):
    """lat: n_xcds lists of latencies; grp: group (0/1) of each XCD."""
    n = len(lat[0])
    members = [[x for x in range(len(grp)) if grp[x] == g] for g in (0, 1)]
    out = []
    for i in range(n):
        m = [sum(lat[x][i] for x in members[g]) / len(members[g]) for g in (0, 1)]
        out.append(-1 if abs(m[0] - m[1]) < tie else (0 if m[0] < m[1] else 1))
    return out


def chunk_homes(page_homes, hash_mask: int, chunk_log2: int):
    in_page = hash_mask & (PAGE - 1)
    if in_page & ((1 << chunk_log2) - 1):
        raise ValueError("the hash has bits below the chunk size")
    per = PAGE >> chunk_log2
    out = []
    for p, h in enumerate(page_homes):
        for c in range(per):
            q = c << chunk_log2
            out.append(-1 if h < 0 else h ^ parity(q & in_page))
    return out


def chunk_lists(home, n_xcds: int, grp, xcd_mask: int, mode: int):
    """Returns (chunk indices XCD by XCD, offsets [n_xcds + 1])."""
    active = [x for x in range(n_xcds) if xcd_mask == 0 or (xcd_mask >> x) & 1]
    if not active:
        raise ValueError("no active XCD")
    per = [[] for _ in range(n_xcds)]
    if mode == ALL:
        for c in range(len(home)):
            per[active[c % len(active)]].append(c)
    else:
        readers = {0: [], 1: []}
        for x in active:
            readers[grp[x] if mode == LOCAL else 1 - grp[x]].append(x)
        dealt = {0: 0, 1: 0}
        for c, h in enumerate(home):
            if h not in (0, 1) or not readers[h]:
                continue
            per[readers[h][dealt[h] % len(readers[h])]].append(c)
            dealt[h] += 1
    out, off = [], []
    for x in range(n_xcds):
        off.append(len(out))
        out.extend(per[x])
    off.append(len(out))
    return out, off
