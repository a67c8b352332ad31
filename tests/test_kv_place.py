"""Page placement for the paged decode-attention cache (host only, no GPU).

The placement is host logic: which pool page holds each (request, head,
32-token page).  The checks restate its contract independently: every entry
is a distinct pool page, with a known home that is the group of the XCD
owning the page's first token's task (LOCAL) or the other group (REMOTE);
IN_ORDER is the dense layout; an inconsistent plan or a pool short of one
group's pages is refused.
"""
import numpy as np
import pytest

import paper_2609_24270_amd as asym

GROUPS = [0, 0, 0, 0, 1, 1, 1, 1]


def plan_of(B, Hkv, S, split, shares):
    n_splits = -(-S // split)
    tasks = B * Hkv * n_splits
    assert sum(shares) == tasks
    return {"split_tokens": split, "n_splits": n_splits, "tasks": tasks, "grid": 8, "tasks_per_workgroup": 4,
            "n_xcds": 8, "tasks_per_xcd": list(shares), "workspace_bytes": 0}


def shares_for(tasks, weights):
    w = np.asarray(weights, dtype=np.float64)
    q = np.floor(tasks * w / w.sum()).astype(int)
    q[: tasks - q.sum()] += 1
    return q.tolist()


def expected_groups(plan, B, Hkv, S, policy):
    pph = -(-S // 32)
    off = np.cumsum([0] + plan["tasks_per_xcd"])
    bh, pg = np.meshgrid(np.arange(B * Hkv), np.arange(pph), indexing="ij")
    task = bh * plan["n_splits"] + (pg * 32) // plan["split_tokens"]
    owner = np.searchsorted(off, task, side="right") - 1
    g = np.asarray(GROUPS)[owner]
    return (g ^ 1 if policy == asym.PAGES_REMOTE else g).reshape(B, Hkv, pph)


@pytest.mark.parametrize("B,Hkv,S,split,weights", [
    (1, 8, 8192, 256, [1] * 8), (2, 8, 1000, 48, [1, 2, 3, 4, 4, 3, 2, 1]), (3, 2, 77, 16, [1] * 8),
    (1, 32, 4096, 1024, [5, 0, 1, 1, 1, 1, 1, 9])])
@pytest.mark.parametrize("policy", [asym.PAGES_LOCAL, asym.PAGES_REMOTE])
def test_local_and_remote_placement(B, Hkv, S, split, weights, policy):
    n_splits = -(-S // split)
    plan = plan_of(B, Hkv, S, split, shares_for(B * Hkv * n_splits, weights))
    pph = -(-S // 32)
    pool_pages = 3 * B * Hkv * pph + 7
    g = np.random.default_rng(S + split)
    home = g.integers(0, 2, size=pool_pages).astype(np.int8)
    home[g.random(pool_pages) < 0.1] = -1  # unknown homes are never used
    t = asym.attn_pages_place(plan, B, Hkv, S, pool_pages, policy, home, GROUPS)
    assert t.shape == (B, Hkv, pph)
    assert len(np.unique(t)) == t.size and t.min() >= 0 and t.max() < pool_pages
    assert np.array_equal(home[t], expected_groups(plan, B, Hkv, S, policy))


def test_in_order_is_the_dense_layout():
    plan = plan_of(2, 4, 100, 32, shares_for(2 * 4 * 4, [1] * 8))
    t = asym.attn_pages_place(plan, 2, 4, 100, 64)
    assert np.array_equal(t.ravel(), np.arange(2 * 4 * 4))


def test_refusals():
    plan = plan_of(1, 8, 1024, 256, shares_for(32, [1] * 8))
    home = np.zeros(1000, dtype=np.int8)  # every page on group 0
    with pytest.raises(asym.AsymError):   # group 1's XCDs need pages homed there
        asym.attn_pages_place(plan, 1, 8, 1024, 1000, asym.PAGES_LOCAL, home, GROUPS)
    with pytest.raises(asym.AsymError):   # the plan is for another sequence length
        asym.attn_pages_place(plan, 1, 8, 2048, 1000, asym.PAGES_LOCAL, home, GROUPS)
    bad = dict(plan, tasks_per_xcd=[4] * 7 + [5])
    mixed = (np.arange(1000) % 2).astype(np.int8)
    assert asym.attn_pages_place(plan, 1, 8, 1024, 1000, asym.PAGES_LOCAL, mixed, GROUPS).size == 256
    with pytest.raises(asym.AsymError):   # shares that do not add up to the tasks
        asym.attn_pages_place(bad, 1, 8, 1024, 1000, asym.PAGES_LOCAL, mixed, GROUPS)
    with pytest.raises(asym.AsymError):   # fewer pool pages than cache pages
        asym.attn_pages_place(plan, 1, 8, 1024, 255)
    with pytest.raises(asym.AsymError):   # homes needed for a placed policy
        asym.attn_pages_place(plan, 1, 8, 1024, 1000, asym.PAGES_LOCAL)
