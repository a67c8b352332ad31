"""GPU parity of decode attention against the float64 oracle, through the C ABI.

Element by element on small shapes covering one and many splits, ragged
sequence tails, a single token, and every supported ratio of query to
key/value heads; on sampled requests at the paper's sizes (32 query heads,
8 or 32 key/value heads, head dimension 128, long sequences).  Bitwise: every
mapping, repeats, a CU-masked stream with unequal CUs per XCD and a whole-XCD
restriction give the same bits (the aware mapping both claiming and, on short
splits over the whole chip, dealing statically).  The plan's task counts follow
the CU counts.
"""
import math

import numpy as np
import pytest
import torch

import paper_2609_24270_amd as asym
from oracle import attention as oat
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


def check(q, k, v, O, lse, scale, what, rows=None):
    qb, kb, vb = bits(q), bits(k), bits(v)
    Ob = bits(O)
    lse_h = lse.cpu().numpy()
    if rows is not None:
        qb, kb, vb, Ob, lse_h = qb[rows], kb[rows], vb[rows], Ob[rows], lse_h[rows]
    R, L = oat.decode_attention(qb, kb, vb, scale)
    err = assert_gemm_close(Ob.reshape(-1, Ob.shape[-1]), R.reshape(-1, R.shape[-1]), what=what)
    lerr = float(np.max(np.abs(lse_h - L) / np.maximum(1.0, np.abs(L))))
    assert lerr < 1e-4, f"{what}: lse rel err {lerr:.3e}"
    return err


@pytest.mark.parametrize("B,Hq,Hkv,S,split", [
    (1, 4, 1, 1, 0), (2, 8, 2, 17, 0), (3, 32, 8, 100, 0), (2, 32, 32, 64, 0), (1, 16, 1, 1000, 0),
    (2, 32, 2, 333, 0), (2, 8, 8, 77, 16), (1, 32, 8, 1000, 48), (2, 16, 8, 4099, 512), (1, 32, 16, 65, 64)])
def test_decode_attention_elementwise(dev, B, Hq, Hkv, S, split):
    p = workloads.AttnProblem(f"t{B}_{Hq}_{Hkv}_{S}", B, Hq, Hkv, S, seed=S + Hq)
    q, k, v = workloads.make_attn_inputs(p)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    O = asym.attn_decode(qd, kd, vd, lse=lse, split_tokens=split)
    torch.cuda.synchronize()
    err = check(q, k, v, O, lse, p.scale, f"B{B} Hq{Hq} Hkv{Hkv} S{S} split{split}")
    assert err < 5e-3


def test_mappings_repeats_and_splits(dev):
    p = workloads.attn_problem("gqa", 4, 3000, seed=21)
    q, k, v = (t.to(dev) for t in workloads.make_attn_inputs(p))
    ref = bits(asym.attn_decode(q, k, v))
    for m in MAPS:
        for _ in range(2):
            assert np.array_equal(bits(asym.attn_decode(q, k, v, mapping=m)), ref), m
    # another split length changes the summation order, not the result beyond rounding
    lse = torch.empty((4, 32), dtype=torch.float32, device=dev)
    O = asym.attn_decode(q, k, v, lse=lse, split_tokens=128)
    torch.cuda.synchronize()
    check(q, k, v, O, lse, p.scale, "split 128")


@pytest.mark.parametrize("kind,B,S", [("gqa", 16, 8192), ("mha", 4, 4096), ("gqa", 64, 2048), ("gqa", 1, 32768)])
def test_paper_sizes_sampled(dev, kind, B, S):
    p = workloads.attn_problem(kind, B, S)
    q, k, v = workloads.make_attn_inputs(p)
    lse = torch.empty((B, 32), dtype=torch.float32, device=dev)
    O = asym.attn_decode(q.to(dev), k.to(dev), v.to(dev), lse=lse)
    torch.cuda.synchronize()
    rows = sorted({0, B // 2, B - 1})
    err = check(q, k, v, O, lse, p.scale, p.name, rows=rows)
    plan = asym.attn_decode_plan(B, 32, p.Hkv, S)
    print(f"{p.name}: sampled max rel err {err:.3e}; split {plan['split_tokens']} x {plan['n_splits']}, "
          f"{plan['tasks']} tasks")


def test_masked_and_restricted_bitwise(dev):
    topo = asym.probe_topology(0, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP)
    p = workloads.attn_problem("gqa", 8, 2048, seed=22)
    q, k, v = (t.to(dev) for t in workloads.make_attn_inputs(p))
    ref = bits(asym.attn_decode(q, k, v))
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    counts = topo.cuset_counts(mask)
    s = asym.stream_create(topo, mask)
    try:
        for m in MAPS:
            plan = asym.attn_decode_plan(8, 32, 8, 2048, mapping=m, topo=topo, stream=s)
            assert sum(plan["tasks_per_xcd"]) == plan["tasks"]
            if m == "aware":
                # proportional to the CU counts, within one task
                for x, c in enumerate(counts):
                    assert abs(plan["tasks_per_xcd"][x] - plan["tasks"] * c / sum(counts)) < 1.0
            O = asym.attn_decode(q, k, v, mapping=m, topo=topo, stream=s)
            s.synchronize()
            assert np.array_equal(bits(O), ref), m
    finally:
        asym.stream_destroy(s)
    for xm in (0x0F, 0x81):
        plan = asym.attn_decode_plan(8, 32, 8, 2048, xcd_mask=xm, topo=topo)
        assert all(plan["tasks_per_xcd"][x] == 0 for x in range(8) if not (xm >> x) & 1)
        O = asym.attn_decode(q, k, v, topo=topo, xcd_mask=xm)
        torch.cuda.synchronize()
        assert np.array_equal(bits(O), ref), hex(xm)


def test_plan_and_rejects(dev):
    plan = asym.attn_decode_plan(1, 32, 8, 512)
    assert plan["split_tokens"] == 64 and plan["n_splits"] == 8 and plan["tasks"] == 64
    plan = asym.attn_decode_plan(64, 32, 8, 32768)
    assert plan["split_tokens"] == 1024 and plan["tasks"] == 64 * 8 * 32
    assert plan["workspace_bytes"] == 64 * 32 * 32 * 130 * 4
    # dense aware calls deal statically only on a uniform set of every XCD, one
    # group per claiming workgroup at most and splits of at most 128 tokens
    assert asym.attn_decode_plan(16, 32, 8, 1024)["dense_static"] == 1
    assert asym.attn_decode_plan(1, 32, 8, 8192)["dense_static"] == 1
    assert asym.attn_decode_plan(16, 32, 8, 8192)["dense_static"] == 0  # 512-token splits
    assert asym.attn_decode_plan(16, 32, 8, 1024, split_tokens=256)["dense_static"] == 0
    assert asym.attn_decode_plan(16, 32, 8, 1024, xcd_mask=0x0F)["dense_static"] == 0
    assert asym.attn_decode_plan(16, 32, 8, 1024, mapping="oblivious_grouped")["dense_static"] == 0
    for kw in (dict(D=64), dict(Hkv=3), dict(split_tokens=20), dict(S=0)):
        args = dict(B=1, Hq=32, Hkv=8, S=128)
        args.update(kw)
        with pytest.raises(asym.AsymError):
            asym.attn_decode_plan(**args)
    with pytest.raises(asym.AsymError):
        asym.attn_decode_plan(1, 32, 8, 128, mapping="oblivious_rowmajor", xcd_mask=0x0F)
    q = torch.zeros((1, 32, 128), dtype=torch.bfloat16, device=dev)
    kv = torch.zeros((1, 8, 64, 128), dtype=torch.bfloat16, device=dev)
    with pytest.raises(asym.AsymError):
        asym.attn_decode(q, kv, kv, scale=math.inf)
