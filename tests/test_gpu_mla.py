"""GPU parity of latent-attention decode against the float64 oracle, through
the C ABI.

Element by element (outputs and log-sum-exp) on small shapes covering one
token, ragged 16-token blocks, one and many splits (automatic and forced),
and 16 to 128 query heads; on sampled (request, head) pairs at the paper's
sizes (long sequences, 128 heads).  Bitwise: every mapping, repeats, a
CU-masked stream with unequal CUs per XCD and whole-XCD restrictions give the
same bits; at multiples of 64 heads both the workgroup form and the wave
form match the oracle.  The plan's task shares follow the CU counts; bad arguments are
refused before any launch.
"""
import numpy as np
import pytest
import torch

import paper_2609_24270_amd as asym
from oracle import mla as omla
from paper_2609_24270_amd import workloads
from tests.checks import assert_gemm_close

pytestmark = pytest.mark.gpu

MAPS = ("aware", "oblivious_grouped", "oblivious_rowmajor")


def bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    asym.load_library()
    torch.cuda.set_device(0)
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def topo(dev):
    return asym.probe_topology(0, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP)


def check(q, kv, O, lse, scale, what, reqs=None, heads=None):
    qb, kb, Ob, lse_h = bits(q), bits(kv), bits(O), lse.detach().cpu().numpy()
    if reqs is not None:
        qb, kb, Ob, lse_h = qb[reqs], kb[reqs], Ob[reqs], lse_h[reqs]
    if heads is not None:
        qb, Ob, lse_h = qb[:, heads], Ob[:, heads], lse_h[:, heads]
    R, L = omla.mla_decode(qb, kb, scale)
    err = assert_gemm_close(Ob.reshape(-1, 512), R.reshape(-1, 512), what=what)
    lerr = float(np.max(np.abs(lse_h - L) / np.maximum(1.0, np.abs(L))))
    assert lerr < 1e-4, f"{what}: lse rel err {lerr:.3e}"
    return err


@pytest.mark.parametrize("B,Hq,S,split", [
    (1, 16, 1, 0), (2, 16, 17, 0), (1, 32, 100, 0), (3, 16, 300, 32), (2, 64, 515, 0), (1, 128, 200, 0),
    (2, 16, 1024, 0), (1, 48, 77, 64), (2, 16, 4111, 1024), (1, 32, 33, 32)])
def test_mla_decode_elementwise(dev, B, Hq, S, split):
    p = workloads.MlaProblem(f"t{B}_{Hq}_{S}", B, Hq, S, seed=S + Hq)
    q, kv = workloads.make_mla_inputs(p)
    qd, kvd = q.to(dev), kv.to(dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    plan = asym.mla_decode_plan(B, Hq, S, split_tokens=split)
    O = asym.mla_decode(qd, kvd, lse=lse, split_tokens=split)
    torch.cuda.synchronize()
    e = check(q, kv, O, lse, p.scale, f"mla B{B} H{Hq} S{S} split {plan['split_tokens']}")
    print(f"mla B{B} H{Hq} S{S}: {plan['n_splits']} splits of {plan['split_tokens']}, max rel err {e:.3e}")


def test_mla_decode_bitwise_across_mappings_masks_and_restrictions(dev, topo):
    p = workloads.MlaProblem("bw", 3, 64, 1500, seed=11)
    q, kv = workloads.make_mla_inputs(p)
    qd, kvd = q.to(dev), kv.to(dev)
    lse = torch.empty((3, 64), dtype=torch.float32, device=dev)
    ref = asym.mla_decode(qd, kvd, lse=lse, topo=topo)
    torch.cuda.synchronize()
    check(q, kv, ref, lse, p.scale, "mla 3x64x1500")
    for m in MAPS:
        for _ in range(2):
            O = asym.mla_decode(qd, kvd, mapping=m, topo=topo)
            torch.cuda.synchronize()
            assert torch.equal(O, ref), m
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    s = asym.stream_create(topo, mask)
    try:
        for m in ("aware", "oblivious_rowmajor"):
            O = asym.mla_decode(qd, kvd, mapping=m, topo=topo, stream=s)
            s.synchronize()
            assert torch.equal(O, ref), ("masked", m)
    finally:
        asym.stream_destroy(s)
    for xm in (0x0F, 0xF0, 0x81):
        O = asym.mla_decode(qd, kvd, topo=topo, xcd_mask=xm)
        torch.cuda.synchronize()
        assert torch.equal(O, ref), hex(xm)
    with pytest.raises(asym.AsymError):
        asym.mla_decode(qd, kvd, mapping="oblivious_grouped", topo=topo, xcd_mask=0x0F)
    # 16 heads (the wave form): the full chip's aware call deals statically,
    # a masked stream and a whole-XCD restriction claim; the same bits
    p = workloads.MlaProblem("bw16", 2, 16, 700, seed=12)
    q, kv = workloads.make_mla_inputs(p)
    qd, kvd = q.to(dev), kv.to(dev)
    assert asym.mla_decode_plan(2, 16, 700, topo=topo)["static_deal"] == 1
    ref = asym.mla_decode(qd, kvd, topo=topo)
    torch.cuda.synchronize()
    s = asym.stream_create(topo, mask)
    try:
        O = asym.mla_decode(qd, kvd, topo=topo, stream=s)
        s.synchronize()
        assert torch.equal(O, ref), "wave form, masked"
    finally:
        asym.stream_destroy(s)
    O = asym.mla_decode(qd, kvd, topo=topo, xcd_mask=0x81)
    torch.cuda.synchronize()
    assert torch.equal(O, ref), "wave form, 0x81"


@pytest.mark.parametrize("B,Hq,S", [(16, 128, 32768), (64, 16, 8192), (4, 128, 65536), (64, 128, 32768),
                                    (8, 128, 16384), (1, 16, 32768)])
def test_mla_decode_paper_sizes_sampled(dev, B, Hq, S):
    p = workloads.mla_problem(B, Hq, S)
    q, kv = workloads.make_mla_inputs_on(p, dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    plan = asym.mla_decode_plan(B, Hq, S)
    if (B, Hq, S) == (64, 128, 32768) and asym.device_query(0)["n_cus"] == 256:
        # the 128-head form with splits lengthened to 4096 tokens (two tasks per CU)
        assert (plan["workgroup_form"], plan["split_tokens"], plan["n_splits"]) == (2, 4096, 8), plan
    if (B, Hq, S) == (8, 128, 16384) and asym.device_query(0)["n_cus"] == 256:
        # the automatic 1024-token split halved for the 128-head form
        assert (plan["workgroup_form"], plan["split_tokens"]) == (2, 512), plan
    if (B, Hq, S) == (1, 16, 32768):
        # 256 splits: 16 waves per row, and the 16 rows' columns cut over 8 merge workgroups
        assert plan["n_splits"] == 256, plan
    O = asym.mla_decode(q, kv, lse=lse)
    torch.cuda.synchronize()
    g = np.random.default_rng(B + Hq)
    reqs = sorted(g.choice(B, size=min(B, 2), replace=False).tolist())
    heads = sorted(g.choice(Hq, size=min(Hq, 6), replace=False).tolist())
    e = check(q[reqs].cpu(), kv[reqs].cpu(), O[reqs].cpu(), lse[reqs].cpu(), p.scale,
              f"mla B{B} H{Hq} S{S} sampled", heads=heads)
    print(f"mla B{B} H{Hq} S{S} sampled requests {reqs} heads {heads}: max rel err {e:.3e}")


def test_mla_plan_shares_and_rejections(dev, topo):
    full = asym.mla_decode_plan(16, 128, 32768, topo=topo)
    # 128 heads: the workgroup form, one task per (request, split, 4 head blocks)
    assert full["head_blocks"] == 8 and full["workgroup_form"] == 2 and full["tasks_per_workgroup"] == 1
    assert full["tasks"] == 16 * full["n_splits"]
    h64 = asym.mla_decode_plan(16, 64, 32768, topo=topo)
    assert h64["workgroup_form"] == 1 and h64["tasks"] == 16 * h64["n_splits"]
    # the 128-head form only where its tasks outnumber half the CUs
    one = asym.mla_decode_plan(1, 128, 32768, topo=topo)
    assert one["workgroup_form"] == 1 and 2 * one["n_splits"] <= 256
    wide = asym.mla_decode_plan(64, 128, 4096, topo=topo)
    assert wide["workgroup_form"] == 2 and 2 * wide["tasks"] > 256
    # an automatic split of 1024 tokens is halved when that lets the 128-head
    # form fill the chip; 512-token splits are not
    mid = asym.mla_decode_plan(8, 128, 16384, topo=topo)
    assert (mid["workgroup_form"], mid["split_tokens"], mid["tasks"]) == (2, 512, 256), mid
    kept = asym.mla_decode_plan(16, 128, 4096, topo=topo)
    assert (kept["workgroup_form"], kept["split_tokens"]) == (1, 512), kept
    small = asym.mla_decode_plan(16, 16, 32768, topo=topo)
    assert small["workgroup_form"] == 0 and small["tasks"] == 16 * small["n_splits"]
    # the static deal: one claiming group per workgroup at most, on a set with
    # equal CUs per XCD over every XCD
    assert wide["static_deal"] == 1 and small["static_deal"] == 1 and one["static_deal"] == 1
    assert full["static_deal"] == 0  # 512 tasks: two per workgroup, the claims balance them
    assert asym.mla_decode_plan(64, 128, 4096, topo=topo, xcd_mask=0x0F)["static_deal"] == 0
    assert asym.mla_decode_plan(64, 128, 4096, mapping="oblivious_grouped", topo=topo)["static_deal"] == 0
    assert sum(full["tasks_per_xcd"]) == full["tasks"] and max(full["tasks_per_xcd"]) - min(full["tasks_per_xcd"]) <= 1
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    counts = topo.cuset_counts(mask)
    s = asym.stream_create(topo, mask)
    try:
        aw = asym.mla_decode_plan(16, 128, 32768, topo=topo, stream=s)
        ob = asym.mla_decode_plan(16, 128, 32768, mapping="oblivious_rowmajor", topo=topo, stream=s)
    finally:
        asym.stream_destroy(s)
    assert aw["static_deal"] == 0
    T = aw["tasks"]
    for x in range(8):
        assert abs(aw["tasks_per_xcd"][x] - T * counts[x] / 128) < 1.0, (x, aw, counts)
    assert max(ob["tasks_per_xcd"]) - min(ob["tasks_per_xcd"]) <= 4
    r = asym.mla_decode_plan(16, 128, 32768, topo=topo, xcd_mask=0x0F)
    assert r["tasks_per_xcd"][4:] == [0] * 4 and sum(r["tasks_per_xcd"]) == r["tasks"]
    for bad in (dict(B=1, Hq=24, S=10), dict(B=0, Hq=16, S=10), dict(B=1, Hq=16, S=10, split_tokens=48)):
        with pytest.raises(asym.AsymError):
            asym.mla_decode_plan(**bad)
    q = torch.zeros((1, 16, 576), dtype=torch.bfloat16, device=dev)
    kv = torch.zeros((1, 8, 576), dtype=torch.bfloat16, device=dev)
    O = torch.zeros((1, 16, 512), dtype=torch.bfloat16, device=dev)
    lib = asym.load_library()
    import ctypes
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    # misaligned output (2 bytes in): refused before any launch
    assert lib.asym_mla_decode_bf16(None, 1, 16, 8, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(kv.data_ptr()),
                                    ctypes.c_void_p(O.data_ptr() + 2), None, 0.1, 0, 0, 0, st) == asym.EINVAL


@pytest.mark.parametrize("B,Hq,S,split", [(2, 64, 515, 0), (1, 128, 200, 0), (3, 128, 1000, 64), (1, 64, 17, 0),
                                          (2, 192, 4111, 1024), (4, 128, 8192, 0), (2, 64, 100, 32),
                                          (2, 256, 333, 0), (1, 128, 31, 32), (2, 128, 4096, 32)])
def test_mla_workgroup_form(dev, topo, B, Hq, S, split):
    """At multiples of 64 heads a workgroup form runs (four head blocks
    sharing each 32-token block of rows through LDS, one softmax step per 32
    tokens, 32-deep P.V products); at multiples of 128 the 128-head form (two
    head blocks per wave, rows loaded straight into LDS), which gives the
    64-head form's bits.  The workgroup forms round differently from the wave
    form (16-token blocks): both are checked against the oracle, on every head
    of the small shapes and on sampled heads of the long ones, and the
    workgroup form's bits are the same on every mapping, on a CU-masked
    stream and under whole-XCD restrictions."""
    p = workloads.MlaProblem(f"wg{B}_{Hq}_{S}", B, Hq, S, seed=S + 3 * Hq)
    q, kv = workloads.make_mla_inputs(p)
    qd, kvd = q.to(dev), kv.to(dev)
    lse_w, lse_g, lse_1 = (torch.empty((B, Hq), dtype=torch.float32, device=dev) for _ in range(3))
    form = 2 if Hq % 128 == 0 else 1
    # level 3: the 128-head form wherever the head count allows (by default it
    # runs only where its tasks fill the CU set, which these small shapes do not)
    prev = asym.set_mla_workgroup_form(3)
    try:
        assert asym.mla_decode_plan(B, Hq, S, split_tokens=split, topo=topo)["workgroup_form"] == form
        got = asym.mla_decode(qd, kvd, lse=lse_g, split_tokens=split, topo=topo)
        torch.cuda.synchronize()
        for m in MAPS[1:]:
            O = asym.mla_decode(qd, kvd, split_tokens=split, mapping=m, topo=topo)
            torch.cuda.synchronize()
            assert torch.equal(O, got), m
        mask = workloads.random_mask_bits(4, 1, 128)[0]
        s = asym.stream_create(topo, mask)
        try:
            O = asym.mla_decode(qd, kvd, split_tokens=split, topo=topo, stream=s)
            s.synchronize()
            assert torch.equal(O, got), "masked"
        finally:
            asym.stream_destroy(s)
        for xm in (0x0F, 0x81):
            O = asym.mla_decode(qd, kvd, split_tokens=split, topo=topo, xcd_mask=xm)
            torch.cuda.synchronize()
            assert torch.equal(O, got), hex(xm)
        asym.set_mla_workgroup_form(1)
        assert asym.mla_decode_plan(B, Hq, S, split_tokens=split, topo=topo)["workgroup_form"] == 1
        form1 = asym.mla_decode(qd, kvd, lse=lse_1, split_tokens=split, topo=topo)
        torch.cuda.synchronize()
        asym.set_mla_workgroup_form(0)
        assert asym.mla_decode_plan(B, Hq, S, split_tokens=split, topo=topo)["workgroup_form"] == 0
        wave = asym.mla_decode(qd, kvd, lse=lse_w, split_tokens=split, topo=topo)
        torch.cuda.synchronize()
    finally:
        asym.set_mla_workgroup_form(prev)
    assert torch.equal(got, form1) and torch.equal(lse_g, lse_1), "128-head form against the 64-head form"
    heads = None if B * Hq * S <= 200_000 else sorted(set([0, Hq - 1, Hq // 2, 17 % Hq]))
    check(q, kv, got, lse_g, p.scale, f"mla workgroup form B{B} H{Hq} S{S}", heads=heads)
    check(q, kv, wave, lse_w, p.scale, f"mla wave form B{B} H{Hq} S{S}", heads=heads)
