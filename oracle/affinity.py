"""Oracle for the XCD-to-memory affinity analysis.  TEST INFRASTRUCTURE ONLY.

Appendix G probes the same sampled addresses from every XCD, groups the XCDs
whose address-dependent latencies move together, and names as an address's
home the group with the lowest mean latency to it; Section 6.1 reads local and
remote latency tiers off the same measurements.  The paper does not say how
"move together" is measured, how groups are formed, or when an address is too
close to call.  Readings taken here:
  * Pearson correlation of two XCDs' per-address latency lists (0 when either
    list is constant);
  * groups = connected components of the graph joining XCDs whose correlation
    is strictly above a threshold, numbered by their lowest XCD;
  * an address's home is the group with the lowest mean latency over its XCDs,
    ties to the lower group number; the address is unclassified when another
    group's mean is less than a tie margin above the lowest (never with one
    group).
Plain Python over lists, exact integer sums; no code shared with the library.
"""
from __future__ import annotations

import math


def pearson(u, v) -> float:
    n = len(u)
    mu = sum(u) / n
    mv = sum(v) / n
    suu = sum((a - mu) * (a - mu) for a in u)
    svv = sum((b - mv) * (b - mv) for b in v)
    if suu == 0 or svv == 0:
        return 0.0
    suv = sum((a - mu) * (b - mv) for a, b in zip(u, v))
    return suv / math.sqrt(suu * svv)


def groups_from_corr(corr, threshold: float):
    n = len(corr)
    label = [-1] * n
    g = 0
    for x in range(n):
        if label[x] >= 0:
            continue
        label[x] = g
        todo = [x]
        while todo:
            u = todo.pop()
            for v in range(n):
                if label[v] < 0 and corr[u][v] > threshold:
                    label[v] = g
                    todo.append(v)
        g += 1
    return label, g


def analyze(lat, threshold: float = 0.5, tie: float = 20.0) -> dict:
    """lat: list of n_xcds lists of n_samples integer latencies."""
    rows = [[int(v) for v in r] for r in lat]
    n_x, n_s = len(rows), len(rows[0])
    corr = [[1.0 if x == y else 0.0 for y in range(n_x)] for x in range(n_x)]
    for x in range(n_x):
        for y in range(x + 1, n_x):
            corr[x][y] = corr[y][x] = pearson(rows[x], rows[y])
    label, n_g = groups_from_corr(corr, threshold)
    members = [[x for x in range(n_x) if label[x] == g] for g in range(n_g)]
    home = []
    for i in range(n_s):
        means = [sum(rows[x][i] for x in m) / len(m) for m in members]
        best = min(range(n_g), key=lambda g: (means[g], g))
        tied = any(g != best and means[g] - means[best] < tie for g in range(n_g))
        home.append(-1 if tied else best)
    share = [home.count(g) / n_s for g in range(n_g)]
    by_home = []
    for x in range(n_x):
        row = []
        for g in range(n_g):
            idx = [i for i in range(n_s) if home[i] == g]
            row.append(sum(rows[x][i] for i in idx) / len(idx) if idx else -1.0)
        by_home.append(row)
    return {"n_xcds": n_x, "n_samples": n_s,
            "hbm": [sum(r) / n_s for r in rows],
            "corr": corr, "group_of_xcd": label, "n_groups": n_g,
            "home": home, "home_share": share,
            "unclassified_share": home.count(-1) / n_s,
            "hbm_by_home": by_home}
