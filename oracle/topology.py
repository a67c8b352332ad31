"""Oracle for the topology map.  TEST INFRASTRUCTURE ONLY.

Section 5.1 recovers which logical units share a physical cluster and Section
5.2 shows the layout differs from chip to chip; the map is therefore whatever
the hardware reports, reduced to a canonical form.  Each identity record holds
the XCC_ID register and the HW_ID register of one workgroup; the GCN/CDNA
HW_ID layout puts the CU id in bits 8-11, the shader array in bit 12 and the
shader engine in bits 13-15.  The map is the sorted list of distinct
(xcc, se, sh, cu) tuples; the dense index of a CU is its position in that list.

Exact invariants (the ones a correct map must satisfy): every CU appears once,
the per-XCD counts sum to the device's CU count, the number of XCDs is the
device's, and a mask-bit map is a bijection between bits and CUs.
"""
from __future__ import annotations


def fields(xcc_reg: int, hw_id: int):
    h = hw_id & 0xFFFFFFFF
    return (xcc_reg & 0xF, (h >> 13) & 0x7, (h >> 12) & 0x1, (h >> 8) & 0xF)


def build_map(records):
    """records: iterable of (xcc_reg, hw_id, block, _) -> sorted distinct tuples."""
    return sorted({fields(r[0], r[1]) for r in records})


def per_xcd_counts(cus, n_xccs: int):
    counts = [0] * n_xccs
    for c in cus:
        counts[c[0]] += 1
    return counts


def invariant_violations(cus, n_cus_device: int, n_xccs_device: int, bit_to_cu=None):
    """List of violated invariants (empty when the map is sound)."""
    bad = []
    if len(set(cus)) != len(cus):
        bad.append("duplicate CU")
    if len(cus) != n_cus_device:
        bad.append("CU count differs from the device's")
    if any(c[0] >= n_xccs_device for c in cus):
        bad.append("XCC id beyond the device's XCC count")
    else:
        counts = per_xcd_counts(cus, n_xccs_device)
        if sum(counts) != n_cus_device:
            bad.append("per-XCD counts do not sum to the CU count")
        if any(v == 0 for v in counts):
            bad.append("an XCD has no CU")
    if bit_to_cu is not None:
        if sorted(bit_to_cu) != list(range(len(cus))) or len(bit_to_cu) != n_cus_device:
            bad.append("mask-bit map is not a bijection")
    return bad


def round_robin_fraction(records, n_xccs: int) -> float:
    """Share of records whose XCC (low 4 bits of the XCC_ID word) is the one
    holding most records of their residue class, block index mod n_xccs.  The
    dealing of workgroups to XCDs is round-robin by block index, but the XCD it
    starts on can differ between launches; what the aware schedules need is
    that each residue class sits on one XCD, which this measures."""
    recs = list(records)
    counts = {}
    for r in recs:
        key = (r[2] % n_xccs, r[0] & 0xF)
        counts[key] = counts.get(key, 0) + 1
    best = {}
    for (cls, x), c in counts.items():
        best[cls] = max(best.get(cls, 0), c)
    return sum(best.values()) / len(recs)
