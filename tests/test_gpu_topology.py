"""GPU tests of the topology probe, CU-masked streams, the copy kernel and co-run.

Topology: the exact invariants (every CU once, per-XCD counts summing to the
device CU count, a bijective mask map whose CUs are the identity probe's CUs).
Masked and XCD-restricted GEMMs must give bitwise the unmasked result.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import topology as otopo
import paper_2609_24270_amd as asym
from paper_2609_24270_amd import workloads
from tests.checks import assert_gemm_close

pytestmark = pytest.mark.gpu


def bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    asym.load_library()
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def topo(dev):
    return asym.probe_topology(0, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP)


def test_identity_probe_invariants(dev):
    t = asym.probe_topology(0, asym.PROBE_IDENTITY)
    d = asym.device_query(0)
    info = t.info()
    cus = [(c["xcc"], c["se"], c["sh"], c["cu"]) for c in t.cus()]
    print("cus_per_xcd", info["cus_per_xcd"], "round-robin fraction", t.dispatch_rr_fraction())
    assert otopo.invariant_violations(cus, d["n_cus"], d["n_xccs"]) == []
    assert info["n_cus"] == d["n_cus"] and sum(info["cus_per_xcd"]) == d["n_cus"]
    assert info["n_xcds"] == d["n_xccs"]


def test_maskmap_probe(dev, topo):
    d = asym.device_query(0)
    cus = topo.cus()
    keys = [(c["xcc"], c["se"], c["sh"], c["cu"]) for c in cus]
    bit_to_cu = [None] * d["n_cus"]
    for i, c in enumerate(cus):
        bit_to_cu[c["mask_bit"]] = i
    assert otopo.invariant_violations(keys, d["n_cus"], d["n_xccs"], bit_to_cu) == []
    ident = asym.probe_topology(0, asym.PROBE_IDENTITY)
    assert keys == [(c["xcc"], c["se"], c["sh"], c["cu"]) for c in ident.cus()]
    js = topo.json()
    print("mask bit -> xcc:", [cus[bit_to_cu[b]]["xcc"] for b in range(32)])
    assert js["has_maskmap"]


def test_dispatch_rule_on_cu_sets(dev, topo):
    """Launches are dealt to XCDs round-robin by block index on the whole chip
    (every residue class of block indices on one XCD); the same check on a
    random 128-CU set and on a striped set reports where masked launches land
    (the aware schedules rely on the rule for locality only).  The XCD that
    dealing starts on is reported for launches that follow launches of 0 to 13
    workgroups."""
    n = asym.device_query(0)["n_cus"]
    rr, per = topo.dispatch_check(None)
    print("full", rr, per)
    assert rr == 1.0 and sum(per) == 4 * n
    for name, m in (("random", workloads.random_mask_bits(4, 1, 128)[0]),
                    ("striped", topo.cuset(128, asym.CUSET_STRIPED))):
        rr, per = topo.dispatch_check(m)
        print(name, rr, per, topo.cuset_counts(m))
        assert 0.0 <= rr <= 1.0 and sum(per) == 4 * n
    rots = {}
    for pre in (0, 1, 3, 8, 13):
        cf, rot, per = topo.dispatch_probe(pre)
        rots[pre] = (round(cf, 4), rot)
        assert cf == 1.0 and sum(per) == 4 * n
    print("after a launch of k workgroups: (class share, rotation)", rots)


def test_masked_gemm_bitwise(dev, topo):
    A, B = workloads.make_inputs(workloads.COLOC)
    Ad, Bd = A.to(dev), B.to(dev)
    ref = asym.gemm(Ad, Bd, mapping="aware")
    torch.cuda.synchronize()
    R, _ = oracle.gemm_bf16(bits(A)[:64], bits(B)[:64], "nk")
    assert_gemm_close(bits(ref)[:64, :64], R)
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    counts = topo.cuset_counts(mask)
    print("random mask per-XCD counts", counts)
    s = asym.stream_create(topo, mask)
    try:
        for m in ("aware", "oblivious_grouped", "oblivious_rowmajor"):
            C = asym.gemm(Ad, Bd, mapping=m, topo=topo, stream=s)
            s.synchronize()
            assert torch.equal(C, ref), m
    finally:
        asym.stream_destroy(s)
    # whole-XCD restriction on an unmasked stream (aware only)
    for xm in (0x0F, 0xF0, 0x81):
        C = asym.gemm(Ad, Bd, mapping="aware", topo=topo, xcd_mask=xm)
        torch.cuda.synchronize()
        assert torch.equal(C, ref), hex(xm)
    with pytest.raises(asym.AsymError):
        asym.gemm(Ad, Bd, mapping="oblivious_grouped", topo=topo, xcd_mask=0x0F)


def test_copy_kernel(dev, topo):
    """The streaming copy on the whole chip, on whole-XCD filters and on a
    CU-masked stream copies every byte, including a size that is not a whole
    number of 16 KiB blocks per XCD; a stop flag raised before the launch ends
    it after one pass; bad arguments are refused."""
    n = workloads.COPY_BYTES // 2
    src = workloads.copy_source(n).to(dev)
    for xm, passes in ((0, 1), (0x3, 2), (0xF0, 3), (0x81, 1)):
        dst = torch.zeros_like(src)
        asym.copy(dst, src, passes=passes, xcd_mask=xm, topo=topo)
        torch.cuda.synchronize()
        assert torch.equal(dst, src), hex(xm)
    s2 = src[: 12345 * 8]
    d2 = torch.zeros_like(s2)
    asym.copy(d2, s2, topo=topo)
    torch.cuda.synchronize()
    assert torch.equal(d2, s2)
    # a seeded random 128-CU set (9 to 23 CUs per XCD) on a masked stream
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    s = asym.stream_create(topo, mask)
    try:
        dst = torch.zeros_like(src)
        asym.copy(dst, src, passes=2, stream=s, topo=topo)
        s.synchronize()
        assert torch.equal(dst, src)
    finally:
        asym.stream_destroy(s)
    def timed(fn):
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        fn()
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1)
    dst = torch.zeros_like(src)
    t10 = timed(lambda: asym.copy(dst, src, passes=10, topo=topo))
    flag = torch.ones(1, dtype=torch.int32, device=dev)
    dst.zero_()
    torch.cuda.synchronize()
    t_flag = timed(lambda: asym.copy(dst, src, passes=1000, stop_flag=flag, topo=topo))
    assert torch.equal(dst, src)
    print("copy of 64 MiB: 10 passes %.3f ms; at most 1000 passes with the stop flag raised %.3f ms"
          % (t10, t_flag))
    assert t_flag < 3 * t10  # the flag ends it after its first pass (1000 passes: ~100 x t10)
    with pytest.raises(asym.AsymError):
        asym.copy(src[1:9], src[:8], topo=topo)      # misaligned source
    with pytest.raises(asym.AsymError):
        asym.copy(src[8:], src[:-8], topo=topo)      # overlapping buffers
    with pytest.raises(asym.AsymError):
        asym.copy(dst, src, passes=0, topo=topo)


def test_corun_gemm_and_copy(dev, topo):
    """A GEMM on a seeded random 128-CU set beside the 64 MiB copy tenant on
    the complementary CUs, and on whole-XCD sides (split masks, each side
    lending one CU per foreign XCD): the GEMM's bits equal its solo run and
    the copy copies every byte; an open-ended copy task is refused."""
    A, B = workloads.make_inputs(workloads.COLOC)
    Ad, Bd = A.to(dev), B.to(dev)
    ref = asym.gemm(Ad, Bd)
    torch.cuda.synchronize()
    C = torch.empty_like(ref)
    src = workloads.copy_source(workloads.COPY_BYTES // 2).to(dev)
    dst = torch.empty_like(src)
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    comp = [b for b in range(256) if b not in set(mask)]
    res = asym.corun([asym.gemm_task(Ad, Bd, C, 5, "aware", mask=mask),
                      asym.copy_task(dst, src, 20, mask=comp)], topo)
    print(res)
    assert torch.equal(C, ref)
    assert torch.equal(dst, src)
    assert res[0]["tflops"] > 0 and res[1]["gbps"] > 0 and res[1]["iters_done"] == 20
    ma, mb = topo.cuset_split_xcds(0x0F)
    dst.zero_()
    C.zero_()
    res = asym.corun([asym.gemm_task(Ad, Bd, C, 5, "aware", mask=ma, xcd_mask=0x0F),
                      asym.copy_task(dst, src, 20, mask=mb, xcd_mask=0xF0)], topo)
    print(res)
    assert torch.equal(C, ref)
    assert torch.equal(dst, src)
    with pytest.raises(asym.AsymError):
        asym.corun([asym.gemm_task(Ad, Bd, C, 1, "aware", mask=mask),
                    asym.copy_task(dst, src, 0, mask=comp)], topo)


def test_corun_prefill_decode(dev, topo):
    """Prefill and decode GEMMs co-running on CU-striped masks (every XCD split
    24/8) and on whole-XCD partitions (6 XCDs / 2 XCDs) give bitwise the
    results of the GEMMs run alone."""
    (pa, pb), (da, db) = workloads.make_pd_inputs()
    pa, pb, da, db = pa.to(dev), pb.to(dev), da.to(dev), db.to(dev)
    ref_p = asym.gemm(pa, pb)
    ref_d = asym.gemm(da, db)
    torch.cuda.synchronize()
    R, _ = oracle.gemm_bf16(bits(da)[:, :], bits(db)[:256], "nk")
    assert_gemm_close(bits(ref_d)[:, :256], R)
    cp = torch.empty_like(ref_p)
    cd = torch.empty_like(ref_d)
    prefill = topo.cuset(192, asym.CUSET_STRIPED)
    decode = [b for b in range(256) if b not in set(prefill)]
    assert topo.cuset_counts(prefill) == [24] * 8 and topo.cuset_counts(decode) == [8] * 8
    res = asym.corun([asym.gemm_task(pa, pb, cp, 3, "aware", mask=prefill),
                      asym.gemm_task(da, db, cd, 20, "aware", mask=decode)], topo)
    print("striped", res)
    assert torch.equal(cp, ref_p) and torch.equal(cd, ref_d)
    assert res[0]["tflops"] > 0 and res[1]["tflops"] > 0
    pm, dm = topo.cuset_split_xcds(0x3F)
    res = asym.corun([asym.gemm_task(pa, pb, cp, 3, "aware", mask=pm, xcd_mask=0x3F),
                      asym.gemm_task(da, db, cd, 20, "aware", mask=dm, xcd_mask=0xC0)], topo)
    print("xcd-aligned", res)
    assert torch.equal(cp, ref_p) and torch.equal(cd, ref_d)
    # with an untimed warm-up of every task first (the timed parts start
    # together once all warm-ups are done): same bits, the timed iterations only
    cp.zero_()
    cd.zero_()
    res = asym.corun([asym.gemm_task(pa, pb, cp, 3, "aware", mask=prefill, warm_iters=30),
                      asym.gemm_task(da, db, cd, 20, "aware", mask=decode, warm_iters=200)], topo)
    print("striped after warm-up", res)
    assert torch.equal(cp, ref_p) and torch.equal(cd, ref_d)
    assert res[0]["iters_done"] == 3 and res[1]["iters_done"] == 20 and res[0]["ms_total"] < 50
    with pytest.raises(asym.AsymError):
        asym.corun([asym.gemm_task(pa, pb, cp, 3, "aware", mask=prefill, warm_iters=-1)], topo)


def test_corun_gemm_with_read_tenant(dev, topo):
    """A GEMM on a seeded random 128-CU set with the bandwidth-bound reader on
    the complementary CUs: the GEMM's bits equal the GEMM run alone for every
    mapping, the reader reports its passes and rate; a read task with no
    passes, or with an XCD filter naming a missing XCD, is refused."""
    A, B = workloads.make_inputs(workloads.COLOC)
    Ad, Bd = A.to(dev), B.to(dev)
    ref = asym.gemm(Ad, Bd)
    torch.cuda.synchronize()
    C = torch.empty_like(ref)
    buf = torch.ones(256 << 20, dtype=torch.float32, device=dev)   # 1 GiB
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    comp = [b for b in range(256) if b not in set(mask)]
    for m in ("aware", "oblivious_grouped", "oblivious_rowmajor"):
        res = asym.corun([asym.gemm_task(Ad, Bd, C, 5, m, mask=mask), asym.read_task(buf, 4, mask=comp)], topo)
        print(m, res)
        assert torch.equal(C, ref), m
        assert res[1]["iters_done"] == 4 and res[1]["gbps"] > 100
    with pytest.raises(asym.AsymError):
        asym.corun([asym.gemm_task(Ad, Bd, C, 1, "aware", mask=mask), asym.read_task(buf, 0, mask=comp)], topo)
    with pytest.raises(asym.AsymError):
        asym.corun([asym.gemm_task(Ad, Bd, C, 1, "aware"), asym.read_task(buf, 1, xcd_mask=0x100)], topo)


def test_corun_tasks_overlap(dev, topo):
    """Co-run tasks run at the same time: a short GEMM on a CU set not used
    before (its schedule is built and uploaded inside the co-run) ends while a
    reader about ten times longer still runs on the complementary CUs.  A
    one-time setup that waited for every stream would start the GEMM only after
    the reader ended."""
    A, B = workloads.make_inputs(workloads.COLOC)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty((A.shape[0], B.shape[0]), dtype=torch.bfloat16, device=dev)
    buf = torch.ones(256 << 20, dtype=torch.float32, device=dev)   # 1 GiB
    for seed in (77, 78):
        mask = workloads.random_mask_bits(seed, 1, 128)[0]
        comp = [b for b in range(256) if b not in set(mask)]
        res = asym.corun([asym.gemm_task(Ad, Bd, C, 3, "aware", mask=mask),
                          asym.read_task(buf, 60, mask=comp)], topo)
        print(seed, res)
        assert res[0]["ms_total"] < 0.5 * res[1]["ms_total"], res


def test_read_tenant_covers_the_buffer(dev, topo):
    """The reader's checksum (XOR of every 16-byte word it read) equals the XOR
    of the buffer's words for an odd pass count: on a CU mask, on the whole
    chip, and with an XCD filter (alone, and on the whole-XCD side of an
    aligned split whose mask lends it one CU on each other XCD, beside a GEMM
    restricted to the other side), on the default grid and on explicit ones
    (more workgroups than the CUs hold; fewer than the XCDs).  A ragged size:
    not a multiple of the per-XCD slices or of the grid's stride."""
    n16 = (48 << 16) + 37
    words = torch.randint(-2**31, 2**31 - 1, (n16 * 4,), dtype=torch.int32,
                          generator=torch.Generator().manual_seed(5))
    want = np.bitwise_xor.reduce(words.numpy().view(np.uint32).reshape(-1, 4), axis=0).tolist()
    buf = words.to(dev)
    A, B = workloads.make_inputs(workloads.COLOC)
    Ad, Bd = A.to(dev), B.to(dev)
    ref = asym.gemm(Ad, Bd)
    torch.cuda.synchronize()
    C = torch.empty_like(ref)
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    comp = [b for b in range(256) if b not in set(mask)]
    cases = [("masked", dict(mask=comp)), ("whole chip", {}), ("xcds 0xF0", dict(xcd_mask=0xF0)),
             ("xcds 0x5A", dict(xcd_mask=0x5A)), ("masked, 3000 workgroups", dict(mask=comp, grid=3000)),
             ("xcds 0x0F, 9 workgroups", dict(xcd_mask=0x0F, grid=9))]
    for name, kw in cases:
        r = asym.corun([asym.read_task(buf, 3, **kw)], topo)
        print(name, r[0]["gbps"], [hex(v) for v in r[0]["checksum"]])
        assert r[0]["checksum"] == want, name
    for xm in (0x0F, 0xF0):
        ma, mb = topo.cuset_split_xcds(xm)
        r = asym.corun([asym.gemm_task(Ad, Bd, C, 5, "aware", mask=ma, xcd_mask=xm),
                        asym.read_task(buf, 3, mask=mb, xcd_mask=0xFF & ~xm)], topo)
        print("aligned", hex(xm), r)
        assert r[1]["checksum"] == want and torch.equal(C, ref), hex(xm)
