"""Oracle for the partition-hash (interleave) discovery.  TEST INFRASTRUCTURE ONLY.

Section 6.1 ("NUMA partition identification"): the memory partition that holds
an address is a hash of its physical address bits, on the GPUs the paper
dissects a single parity (XOR) over a subset of them.  Flipping one bit of an
address and checking, by latency, whether the address changes partition tells
whether that bit takes part; the lowest bit that takes part sets the
granularity, the largest aligned range that always stays in one partition.

Here an address's partition is its home affinity group from the latency
analysis (oracle.affinity.analyze: groups of XCDs by correlated HBM
latencies, home = the group with the lowest mean latency).  Readings taken
where the paper gives no rule:
  * the addresses come in blocks of equal size: a base line first, then
    variants of the base with one or two offset bits flipped.  The flipped bits
    are read from the XOR of a variant's offset with its base's, so the
    analysis needs no other description of the layout;
  * a bit's flip fraction is, over the blocks where the base and its one-bit
    variant both have a home, the share whose homes differ.  The bit takes
    part (verdict 1) when the fraction is at least 1 - decide, does not
    (verdict 0) when it is at most decide, and is undetermined (-1) otherwise
    or when no block has both homes; a bit no variant flips is untested (-2).
    A bit above the translation page flips a virtual address onto another
    physical page and lands undetermined unless the pages are contiguous;
  * a two-bit variant checks linearity: under one parity its home differs from
    the base's exactly when one of the two bits takes part.  Only pairs whose
    two bits have verdict 0 or 1 and whose two homes exist are counted;
  * the granularity is 2 to the lowest participating bit, when every tested bit
    below it has a verdict; else unknown;
  * the local and remote tiers are the mean latencies over (XCD, address) pairs
    whose address has a home in the XCD's own group, or in another group.
Plain Python; no code shared with the library.
"""
from __future__ import annotations

from . import affinity

NOT_TESTED, UNDETERMINED = -2, -1


def _bits(x: int):
    out, b = [], 0
    while x:
        if x & 1:
            out.append(b)
        x >>= 1
        b += 1
    return out


def analyze(lat, offs, block: int, threshold: float = 0.5, tie: float = 20.0,
            decide: float = 0.1) -> dict:
    """lat: n_xcds lists of per-address HBM latencies; offs: byte offsets of the
    addresses, in blocks of `block` (base first)."""
    n_addr = len(offs)
    if block < 1 or n_addr % block:
        raise ValueError("addresses must come in whole blocks")
    a = affinity.analyze(lat, threshold, tie)
    home = a["home"]
    usable = [0] * 64
    flips = [0] * 64
    tested = [False] * 64
    pairs = []
    for b0 in range(0, n_addr, block):
        for j in range(b0 + 1, b0 + block):
            d = _bits(offs[j] ^ offs[b0])
            if len(d) == 1:
                i = d[0]
                tested[i] = True
                if home[b0] >= 0 and home[j] >= 0:
                    usable[i] += 1
                    flips[i] += home[b0] != home[j]
            elif len(d) == 2:
                pairs.append((b0, j, d[0], d[1]))
    frac = [flips[i] / usable[i] if usable[i] else -1.0 for i in range(64)]
    verdict = []
    for i in range(64):
        if not tested[i]:
            verdict.append(NOT_TESTED)
        elif usable[i] == 0:
            verdict.append(UNDETERMINED)
        elif frac[i] >= 1.0 - decide:
            verdict.append(1)
        elif frac[i] <= decide:
            verdict.append(0)
        else:
            verdict.append(UNDETERMINED)
    checks = agree = 0
    for b0, j, i, k in pairs:
        if verdict[i] in (0, 1) and verdict[k] in (0, 1) and home[b0] >= 0 and home[j] >= 0:
            checks += 1
            agree += (home[b0] != home[j]) == ((verdict[i] ^ verdict[k]) == 1)
    mask = sum(1 << i for i in range(64) if verdict[i] == 1)
    lowest = min((i for i in range(64) if verdict[i] == 1), default=-1)
    tested_bits = [i for i in range(64) if tested[i]]
    undet = [i for i in tested_bits if verdict[i] == UNDETERMINED]
    determined_below = min(undet) if undet else (max(tested_bits) + 1 if tested_bits else 0)
    gran = (1 << lowest) if 0 <= lowest < determined_below else -1
    grp = a["group_of_xcd"]
    loc = [lat[x][i] for x in range(len(lat)) for i in range(n_addr) if home[i] >= 0 and home[i] == grp[x]]
    rem = [lat[x][i] for x in range(len(lat)) for i in range(n_addr) if home[i] >= 0 and home[i] != grp[x]]
    return {"local_cycles": sum(loc) / len(loc) if loc else -1.0,
            "remote_cycles": sum(rem) / len(rem) if rem else -1.0,
            "n_groups": a["n_groups"], "group_of_xcd": a["group_of_xcd"], "home": home,
            "unclassified_share": a["unclassified_share"],
            "flip_fraction": frac, "usable": usable, "verdict": verdict,
            "hash_mask": mask, "lowest_bit": lowest, "determined_below": determined_below,
            "granularity": gran, "pair_checks": checks, "pair_agree": agree,
            "linear_consistency": agree / checks if checks else -1.0}
