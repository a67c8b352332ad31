"""GPU parity of the paged decode attention, through the C ABI.

The paged form reads the same keys and values as the dense form, only from
other addresses, so its outputs and log-sum-exp must be bitwise those of the
dense call (itself element-wise green against the float64 oracle), for
random page tables, for placements computed by the host (local and remote to
the reading XCD's die, on made-up page homes: correctness does not depend on
the homes), for tables naming one page twice, ragged sequence ends, splits
of 16 tokens past a page boundary and of 2048 tokens, GQA ratios 1 to 16, every
mapping and a whole-XCD restriction.  Pool pages no entry names are filled
with large values, so a read of a wrong page changes the result.  One case at
a paper size (B = 1, S = 32768) is also checked against the oracle on sampled
heads.
"""
import numpy as np
import pytest
import torch

import paper_2609_24270_amd as asym
from oracle import attention as oatt
from paper_2609_24270_amd import workloads
from tests.checks import assert_gemm_close

pytestmark = pytest.mark.gpu

GROUPS = [0, 0, 0, 0, 1, 1, 1, 1]


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    asym.load_library()
    torch.cuda.set_device(0)
    return torch.device("cuda:0")


def dense_and_paged(dev, B, Hq, Hkv, S, split=0, mapping="aware", xcd_mask=0, table=None, seed=0):
    """Dense and paged calls on the same inputs.  K and V get independent
    random tables unless `table` is given (then both use it)."""
    p = workloads.AttnProblem(f"paged_{B}_{Hq}_{Hkv}_{S}", B, Hq, Hkv, S, seed=seed + S)
    q, k, v = workloads.make_attn_inputs(p)
    qd, kd, vd = q.to(dev), k.to(dev), v.to(dev)
    pph = -(-S // 32)
    n = B * Hkv * pph
    pool_pages = 2 * n + 5
    if table is None:
        g = np.random.default_rng(seed + 1)
        kt_h = g.permutation(pool_pages)[:n].reshape(B, Hkv, pph).astype(np.int32)
        vt_h = g.permutation(pool_pages)[:n].reshape(B, Hkv, pph).astype(np.int32)
    else:
        pool_pages = max(pool_pages, int(table.max()) + 1)
        kt_h = vt_h = table
    kt = torch.as_tensor(kt_h, dtype=torch.int32).to(dev).contiguous()
    vt = torch.as_tensor(vt_h, dtype=torch.int32).to(dev).contiguous()
    kp = workloads.page_pool(kd, kt, pool_pages, fill=300.0)
    vp = workloads.page_pool(vd, vt, pool_pages, fill=-300.0)
    l1 = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    l2 = torch.empty_like(l1)
    ref = asym.attn_decode(qd, kd, vd, lse=l1, split_tokens=split, mapping=mapping, xcd_mask=xcd_mask)
    got = asym.attn_decode_paged(qd, kp, vp, kt, vt, S, lse=l2, split_tokens=split, mapping=mapping,
                                 xcd_mask=xcd_mask)
    torch.cuda.synchronize()
    return (q, k, v), ref, got, l1, l2


@pytest.mark.parametrize("B,Hq,Hkv,S,split", [
    (1, 32, 8, 1000, 0), (2, 32, 32, 77, 0), (3, 16, 1, 4111, 0), (1, 32, 8, 3000, 48), (2, 8, 8, 5000, 2048),
    (1, 32, 16, 33, 16), (4, 32, 8, 2048, 256)])
def test_paged_equals_dense_bitwise(dev, B, Hq, Hkv, S, split):
    _, ref, got, l1, l2 = dense_and_paged(dev, B, Hq, Hkv, S, split)
    assert torch.equal(got, ref) and torch.equal(l1, l2), (B, Hq, Hkv, S, split)


@pytest.mark.parametrize("mapping,xcd_mask", [("oblivious_grouped", 0), ("oblivious_rowmajor", 0), ("aware", 0x0F),
                                              ("aware", 0x81)])
def test_paged_mappings_and_restrictions(dev, mapping, xcd_mask):
    _, ref, got, l1, l2 = dense_and_paged(dev, 2, 32, 8, 2500, mapping=mapping, xcd_mask=xcd_mask, seed=3)
    assert torch.equal(got, ref) and torch.equal(l1, l2)


@pytest.mark.parametrize("policy", [asym.PAGES_IN_ORDER, asym.PAGES_LOCAL, asym.PAGES_REMOTE])
def test_host_placements(dev, policy):
    B, Hq, Hkv, S = 1, 32, 8, 8192
    plan = asym.attn_decode_plan(B, Hq, Hkv, S)
    pph = S // 32
    pool_pages = 3 * B * Hkv * pph
    home = (np.random.default_rng(5).random(pool_pages) < 0.5).astype(np.int8)
    table = asym.attn_pages_place(plan, B, Hkv, S, pool_pages, policy, home, GROUPS)
    _, ref, got, l1, l2 = dense_and_paged(dev, B, Hq, Hkv, S, table=table, seed=4)
    assert torch.equal(got, ref) and torch.equal(l1, l2)


def test_one_page_named_twice(dev):
    """Every entry names pool page 0: the dense equivalent repeats page 0's
    32 tokens along the sequence."""
    B, Hq, Hkv, S = 1, 8, 2, 300
    g = torch.Generator().manual_seed(9)
    q = torch.randn((B, Hq, 128), generator=g).to(torch.bfloat16)
    page_k = torch.randn((32, 128), generator=g).to(torch.bfloat16)
    page_v = torch.randn((32, 128), generator=g).to(torch.bfloat16)
    pool_k = torch.stack([page_k, torch.full_like(page_k, 300.0)]).to(dev)
    pool_v = torch.stack([page_v, torch.full_like(page_v, -300.0)]).to(dev)
    t = torch.zeros((B, Hkv, -(-S // 32)), dtype=torch.int32, device=dev)
    rep = lambda pg: pg.repeat(-(-S // 32), 1)[:S].expand(B, Hkv, S, 128).contiguous()
    ref = asym.attn_decode(q.to(dev), rep(page_k).to(dev), rep(page_v).to(dev))
    got = asym.attn_decode_paged(q.to(dev), pool_k, pool_v, t, t, S)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)


def test_paper_size_against_the_oracle(dev):
    """B = 1, GQA 32 / 8, S = 32768 with a local placement: sampled heads
    against the float64 oracle."""
    B, Hq, Hkv, S = 1, 32, 8, 32768
    plan = asym.attn_decode_plan(B, Hq, Hkv, S)
    pph = S // 32
    pool_pages = 2 * B * Hkv * pph + 64
    home = (np.arange(pool_pages) % 2).astype(np.int8)
    table = asym.attn_pages_place(plan, B, Hkv, S, pool_pages, asym.PAGES_LOCAL, home, GROUPS)
    (q, k, v), ref, got, l1, l2 = dense_and_paged(dev, B, Hq, Hkv, S, table=table, seed=8)
    assert torch.equal(got, ref) and torch.equal(l1, l2)
    heads = [0, 5, 17, 31]
    bits = lambda t: t.contiguous().view(torch.int16).numpy().view(np.uint16)
    # one query head per sampled head, against its own key/value head
    R, L = oatt.decode_attention(bits(q[:, heads]), bits(k[:, [h // 4 for h in heads]]),
                                 bits(v[:, [h // 4 for h in heads]]), 1.0 / np.sqrt(128))
    e = assert_gemm_close(bits(got.cpu()[:, heads]).reshape(-1, 128), R.reshape(-1, 128), what="paged S=32768")
    lerr = float(np.max(np.abs(l2.cpu().numpy()[:, heads] - L) / np.maximum(1.0, np.abs(L))))
    assert lerr < 1e-4, lerr
    print(f"paged B1 S32768 local placement: max rel err {e:.3e} on heads {heads}")


def test_paged_rejections(dev):
    q = torch.zeros((1, 8, 128), dtype=torch.bfloat16, device=dev)
    pool = torch.zeros((4, 32, 128), dtype=torch.bfloat16, device=dev)
    t = torch.zeros((1, 8, 2), dtype=torch.int32, device=dev)
    t65 = torch.zeros((1, 8, 65), dtype=torch.int32, device=dev)
    with pytest.raises(asym.AsymError):  # splits above 2048 tokens
        asym.attn_decode_paged(q, pool, pool, t65, t65, 2080, split_tokens=2064)
    with pytest.raises(ValueError):  # table shape must match S
        asym.attn_decode_paged(q, pool, pool, t, t, 100)
    import ctypes
    lib = asym.load_library()
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    o = torch.empty((1, 8, 128), dtype=torch.bfloat16, device=dev)
    args = lambda kp, vp, pages: (None, 1, 8, 8, 40, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(pool.data_ptr()),
                                  ctypes.c_void_p(pool.data_ptr()), pages, kp, vp, ctypes.c_void_p(o.data_ptr()),
                                  None, 0.1, 0, 0, 0, st)
    tp = ctypes.c_void_p(t.data_ptr())
    assert lib.asym_attn_decode_paged_bf16(*args(None, tp, 4)) == asym.EINVAL
    assert lib.asym_attn_decode_paged_bf16(*args(tp, tp, 0)) == asym.EINVAL
    assert lib.asym_attn_decode_paged_bf16(*args(tp, tp, (1 << 18) + 1)) == asym.EINVAL
    assert lib.asym_attn_decode_paged_bf16(*args(ctypes.c_void_p(t.data_ptr() + 2), tp, 4)) == asym.EINVAL
