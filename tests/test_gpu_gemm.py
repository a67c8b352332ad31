"""GPU parity of the persistent bf16 GEMM against the CPU oracle.

All calls go through libasym's C ABI.  Small shapes are compared element by
element; full-size shapes (8192^3 and the decoder projections) on sampled rows
and columns, which the oracle computes as a sub-GEMM.  Bitwise properties that
hold at any size: every mapping, CU mask and repeat gives identical bits, and
exact-integer inputs give exactly the integer product.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_24270_amd as asym
from paper_2609_24270_amd import workloads
from tests.checks import REL_TOL, assert_gemm_close

pytestmark = pytest.mark.gpu

MAPS = ("aware", "oblivious_grouped", "oblivious_rowmajor")


def bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    asym.load_library()
    torch.cuda.set_device(0)
    return torch.device("cuda:0")


def run(A, B, mapping="aware", stream=None, **kw):
    C = asym.gemm(A, B, mapping=mapping, stream=stream, **kw)
    torch.cuda.synchronize()
    return C


def sampled_check(A, B, C, n_rows=128, n_cols=128, seed=0, exact=False):
    g = np.random.default_rng(seed)
    M, N = C.shape
    rows = np.sort(g.choice(M, size=min(n_rows, M), replace=False))
    cols = np.sort(g.choice(N, size=min(n_cols, N), replace=False))
    # always include the last row / column (ragged tile edges)
    rows[-1], cols[-1] = M - 1, N - 1
    rows, cols = np.unique(rows), np.unique(cols)
    Ab, Bb, Cb = bits(A), bits(B), bits(C)
    R, Co = oracle.gemm_bf16(Ab[rows], Bb[cols], "nk")
    got = Cb[np.ix_(rows, cols)]
    if exact:
        assert np.array_equal(got, Co)
        return 0.0
    return assert_gemm_close(got, R)


def test_device_query(dev):
    """Device discovery: counts, the chip's identity and its partition modes
    (recorded; SPX / NPS1 expected, "unknown" where the driver's files cannot
    be read), and the cache key that ties a probe result to them."""
    d = asym.device_query(0)
    print(d)
    assert d["n_cus"] == 256 and d["n_xccs"] == 8 and d["arch"].startswith("gfx950")
    assert len(d["uuid"]) == 32 and d["pci_bus_id"].count(":") == 2
    assert d["compute_partition"] and d["memory_partition"]
    key = asym.topology_cache_key(0)
    print("cache key:", key)
    for part in ("pci=" + d["pci_bus_id"], "uuid=" + d["uuid"], "compute=" + d["compute_partition"],
                 "memory=" + d["memory_partition"], "cus=256", "xccs=8"):
        assert part in key, part


def test_topology_cache_on_the_device(dev, tmp_path):
    """The first probe with a cache path probes and writes the file; the
    second reuses it (no probe: same map, same key); a request for a probe the
    file lacks probes again and rewrites it."""
    import time
    path = str(tmp_path / "topo_cache.txt")
    t0 = time.perf_counter()
    a = asym.probe_topology(0, asym.PROBE_IDENTITY, cache_path=path)
    t1 = time.perf_counter()
    b = asym.probe_topology(0, asym.PROBE_IDENTITY, cache_path=path)
    t2 = time.perf_counter()
    ja, jb = a.json(), b.json()
    print("probe %.3f s, cached %.3f s; partitions %s / %s" % (t1 - t0, t2 - t1, ja["compute_partition"],
                                                              ja["memory_partition"]))
    assert ja["cus"] == jb["cus"] and ja["key"] == jb["key"] == asym.topology_cache_key(0)
    assert ja["compute_partition"] == asym.device_query(0)["compute_partition"]
    c = asym.probe_topology(0, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP, cache_path=path)
    assert c.json()["has_maskmap"]
    d = asym.topology_load(path, asym.topology_cache_key(0), asym.PROBE_MASKMAP)
    assert d.json()["cus"] == c.json()["cus"]


@pytest.mark.parametrize("mapping", MAPS)
def test_gemm_512_parity(dev, mapping):
    A, B = workloads.make_inputs(workloads.SQUARE_512)
    R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
    C = run(A.to(dev), B.to(dev), mapping)
    e = assert_gemm_close(bits(C), R, what=f"512^3 {mapping}")
    print(f"512^3 {mapping}: max rel err {e:.3e}")


def test_gemm_mappings_and_repeats_bitwise(dev):
    A, B = workloads.make_inputs(workloads.SQUARE_512)
    A, B = A.to(dev), B.to(dev)
    ref = bits(run(A, B, "aware"))
    for m in MAPS:
        for _ in range(2):
            assert np.array_equal(bits(run(A, B, m)), ref), m


ODD = [(1, 1, 1), (17, 17, 17), (129, 1000, 17), (1000, 129, 129), (17, 1, 1000), (1, 1000, 129),
       (300, 520, 72), (257, 255, 64), (513, 1031, 200), (32, 14336, 4096), (100, 300, 4104)]


@pytest.mark.parametrize("M,N,K", ODD)
def test_gemm_odd_shapes(dev, M, N, K):
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=M + 3 * N + 7 * K))
    R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
    for m in ("aware", "oblivious_grouped"):
        C = run(A.to(dev), B.to(dev), m)
        assert_gemm_close(bits(C), R, what=f"{M}x{N}x{K} {m}")


def test_gemm_strided_and_unaligned(dev):
    # leading dimensions larger than the row, and a K that is not a multiple of 8
    M, N, K = 200, 136, 150
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=9))
    R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
    Ap = torch.zeros((M, K + 24), dtype=torch.bfloat16)
    Ap[:, :K] = A
    Bp = torch.zeros((N, K + 40), dtype=torch.bfloat16)
    Bp[:, :K] = B
    Cp = torch.full((M, N + 8), 7.0, dtype=torch.bfloat16, device=dev)
    asym.gemm(Ap.to(dev)[:, :K], Bp.to(dev)[:, :K], Cp[:, :N])
    torch.cuda.synchronize()
    assert_gemm_close(bits(Cp[:, :N]), R)
    # the padding columns of C are untouched
    assert torch.all(Cp[:, N:].cpu() == 7.0)


def test_gemm_128_tiles_equal_256_tiles_bitwise(dev):
    """The 128 x 128 tiles of a small product give bitwise the outputs the
    256 x 256 tiles give for the same rows and columns of a larger product
    with the same K (each output is the same MFMA chain): on the vector path
    (K multiple of 8) and on the predicated path (K = 1000 + 4)."""
    for K, big in ((1024, 4096), (1004, 2304)):
        A, B = workloads.make_inputs(workloads.make_problem(big, big, K, seed=K))
        Ad, Bd = A.to(dev), B.to(dev)
        assert asym.gemm_plan(Ad, Bd)["tile_m"] == 256
        assert asym.gemm_plan(Ad[:512], Bd[:384])["tile_m"] == 128
        C_big = asym.gemm(Ad, Bd)
        C_small = asym.gemm(Ad[:512].contiguous(), Bd[:384].contiguous())
        torch.cuda.synchronize()
        assert torch.equal(C_small, C_big[:512, :384]), K
        R, _ = oracle.gemm_bf16(bits(A[:512]), bits(B[:384]), "nk")
        assert_gemm_close(bits(C_small), R, what=f"128 tiles, K={K}")


@pytest.mark.parametrize("M,N,K", [(512, 512, 512), (300, 520, 264), (129, 1000, 77), (32, 4096, 4096),
                                   (1000, 136, 2056)])
def test_gemm_b_stored_kn_equals_nk(dev, M, N, K):
    """B stored [K][N] (N contiguous) is transposed into the library's buffer
    and gives bitwise the product of the same logical B stored [N][K], on the
    persistent kernel (vector and predicated paths) and the small-M kernel;
    a [K][N] operand with a leading dimension above N works too."""
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=31 + M + N + K))
    Ad, Bd = A.to(dev), B.to(dev)
    ref = asym.gemm(Ad, Bd)
    Bkn = Bd.t().contiguous()
    assert asym.gemm_plan(A=Ad, B=Bkn, b_layout="kn")["b_transposed"] == 1
    assert asym.gemm_plan(A=Ad, B=Bd)["b_transposed"] == 0
    for m in ("aware", "oblivious_rowmajor"):
        C = asym.gemm(Ad, Bkn, mapping=m, b_layout="kn")
        torch.cuda.synchronize()
        assert torch.equal(C, ref), m
    wide = torch.zeros((K, N + 24), dtype=torch.bfloat16, device=dev)
    wide[:, :N] = Bkn
    C = asym.gemm(Ad, wide[:, :N], b_layout="kn")
    torch.cuda.synchronize()
    assert torch.equal(C, ref)
    R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
    assert_gemm_close(bits(C), R, what=f"[K][N] {M}x{N}x{K}")


def test_gemm_exact_integer_8192_sampled(dev):
    p = workloads.make_problem(8192, 8192, 8192, seed=21, dist="int")
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    C = run(Ad, Bd, "aware")
    sampled_check(A, B, C, 96, 96, seed=1, exact=True)
    C2 = run(Ad, Bd, "oblivious_grouped")
    assert torch.equal(C, C2)


def test_gemm_8192_uniform_sampled(dev):
    A, B = workloads.make_inputs(workloads.SQUARE_8192)
    Ad, Bd = A.to(dev), B.to(dev)
    C = run(Ad, Bd, "aware")
    e = sampled_check(A, B, C, 128, 128, seed=2)
    print(f"8192^3 aware sampled max rel err {e:.3e}")
    for m in ("oblivious_grouped", "oblivious_rowmajor"):
        assert torch.equal(run(Ad, Bd, m), C), m


@pytest.mark.parametrize("p", workloads.LLM_SHAPES, ids=lambda p: p.name)
def test_gemm_llm_shapes_sampled(dev, p):
    A, B = workloads.make_inputs(p)
    C = run(A.to(dev), B.to(dev), "aware")
    e = sampled_check(A, B, C, 128, 128, seed=3)
    print(f"{p.name} sampled max rel err {e:.3e}")


# Tile widths: the launch takes 256, 224 or 192 columns per tile, whichever
# leaves the persistent workers the fewest rounds of tiles.  With the aware
# grid kept to XCD 0 (32 workers) and two tile rows, each width is the choice
# for one of these shapes, every one with ragged M, N and K tails.
WIDTH_CASES = [(256, 500, 4092, 328), (224, 500, 3548, 328), (192, 500, 1100, 328)]


@pytest.mark.parametrize("width,M,N,K", WIDTH_CASES, ids=lambda v: str(v))
def test_gemm_tile_widths_elementwise(dev, width, M, N, K):
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=width + N))
    Ad, Bd = A.to(dev), B.to(dev)
    plan = asym.gemm_plan(Ad, Bd, mapping="aware", xcd_mask=1)
    assert plan["tile_n"] == width and plan["vector_path"] == 1, plan
    assert plan["workers"] == 32 and plan["workers_per_xcd"][1:] == [0] * 7, plan
    R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
    C = run(Ad, Bd, "aware", xcd_mask=1)
    e = assert_gemm_close(bits(C), R, what=f"width {width} {M}x{N}x{K}")
    print(f"width {width} {M}x{N}x{K}: max rel err {e:.3e}")
    # other tiles over the whole chip (128 x 128: these products have too few
    # 256-row tiles for 256 workers) give the same bits
    full = asym.gemm_plan(Ad, Bd, mapping="aware")
    assert (full["tile_m"], full["tile_n"]) == (128, 128) and full["workers"] == 256, full
    assert torch.equal(run(Ad, Bd, "aware"), C)


def test_gemm_plan_full_sizes(dev):
    """The widths and forms the full-size workloads launch with."""
    want = {(8192, 8192, 8192): 256, (4096, 14336, 4096): 224, (4096, 4096, 14336): 256,
            (4096, 6144, 4096): 192}
    for (M, N, K), w in want.items():
        for m in MAPS:
            p = asym.gemm_plan(mapping=m, M=M, N=N, K=K)
            assert p["tile_m"] == 256 and p["tile_n"] == w, (M, N, K, m, p)
            assert p["tiles_m"] == -(-M // 256) and p["tiles_n"] == -(-N // w)
            assert p["workers"] == 256 and p["workers_per_xcd"] == [32] * 8
            assert p["claims"] == 0
            assert p["grid"] == 256
    # a whole-XCD restriction takes claims (workers read XCC_ID)
    p = asym.gemm_plan(mapping="aware", M=8192, N=8192, K=8192, xcd_mask=0x0F)
    assert p["claims"] == 1 and p["workers"] == 128 and p["workers_per_xcd"] == [32] * 4 + [0] * 4
    # the predicated path keeps the 256-wide tile
    p = asym.gemm_plan(mapping="aware", M=2304, N=2304, K=150)
    assert p["vector_path"] == 0 and (p["tile_m"], p["tile_n"]) == (256, 256)
    # products whose 256 x 256 tiles would leave 3/4 of the workers idle take 128 x 128 tiles
    for (M, N, K) in ((512, 512, 512), (300, 700, 150), (2048, 2048, 1024), (129, 1000, 77)):
        p = asym.gemm_plan(mapping="aware", M=M, N=N, K=K)
        assert (p["tile_m"], p["tile_n"]) == (128, 128), (M, N, K, p)
        assert (p["tiles_m"], p["tiles_n"]) == (-(-M // 128), -(-N // 128))
    p = asym.gemm_plan(mapping="aware", M=512, N=512, K=512, xcd_mask=0x01)      # 32 workers
    assert (p["tile_m"], p["tiles_m"], p["tiles_n"]) == (128, 4, 4)
    assert asym.gemm_plan(mapping="aware", M=2304, N=2048, K=1024)["tile_m"] == 256


def test_gemm_plan_rejects_like_launch(dev):
    with pytest.raises(asym.AsymError) as e:
        asym.gemm_plan(M=0, N=8, K=8)
    assert e.value.status == asym.EINVAL
    with pytest.raises(asym.AsymError) as e:
        asym.gemm_plan(mapping="oblivious_grouped", M=64, N=64, K=64, xcd_mask=1)
    assert e.value.status == asym.EUNSUPPORTED


# k-stage isolation: with A (or B) zero outside one 64-wide k stage, C is that
# stage's product alone, so a stage read from the wrong ring slot, or data
# landing in the wrong slot, shows up as a wrong stage.  Small integers make
# the fp32 sums exact, so the output must equal the oracle's bit for bit.
# Each tile width, with stage counts that are not multiples of the ring's
# three A slots; XCD 0 only (32 workers) so that the widths are the chosen ones.
# The last three give each of the 32 workgroups two tiles (the rings run on
# from one tile into the next), with K of 7 stages, of 2 (the fewest that run
# on) and of 1 (each tile starts with its own prologue).
STAGE_CASES = [(256, 500, 4092, 7), (224, 500, 3548, 5), (192, 500, 1100, 8),
               (256, 1000, 4092, 7), (256, 1000, 4092, 2), (256, 1000, 4092, 1)]


@pytest.mark.parametrize("width,M,N,KT", STAGE_CASES, ids=lambda v: str(v))
def test_gemm_ring_stage_isolation(dev, width, M, N, KT):
    K = 64 * KT
    g = np.random.default_rng(width + KT)
    A = g.integers(-3, 4, size=(M, K)).astype(np.float32)
    B = g.integers(-3, 4, size=(N, K)).astype(np.float32)
    assert asym.gemm_plan(M=M, N=N, K=K, xcd_mask=1)["tile_n"] == width
    for which in ("A", "B"):
        for s in range(KT):
            a, b = A.copy(), B.copy()
            x = a if which == "A" else b
            x[:, :64 * s] = 0
            x[:, 64 * s + 64:] = 0
            ta = torch.tensor(a, dtype=torch.bfloat16)
            tb = torch.tensor(b, dtype=torch.bfloat16)
            _, ref = oracle.gemm_bf16(bits(ta), bits(tb), "nk")
            C = run(ta.to(dev), tb.to(dev), "aware", xcd_mask=1)
            assert np.array_equal(bits(C), ref), f"width {width}: {which} stage {s} of {KT}"


def test_gemm_trace_records(dev):
    """The traced launch gives the bits of the untraced one and one record per
    workgroup: every tile computed once in all, on the XCC each record names,
    within the launch's time span; on the full chip (static aware form) every
    worker computes its region's share; under a whole-XCD restriction only the
    chosen XCDs' workgroups work."""
    topo = asym.probe_topology(0, asym.PROBE_IDENTITY)
    A, B = workloads.make_inputs(workloads.make_problem(4096, 4096, 1024, seed=77))
    Ad, Bd = A.to(dev), B.to(dev)
    ref = asym.gemm(Ad, Bd, topo=topo)
    C = torch.zeros_like(ref)
    t = asym.gemm_trace(Ad, Bd, C, topo=topo)
    assert torch.equal(C, ref)
    T = t["plan"]["tiles_m"] * t["plan"]["tiles_n"]
    assert len(t["tiles"]) == t["plan"]["grid"] == 256 and int(t["tiles"].sum()) == T == 256
    assert set(t["xcc"].tolist()) <= set(range(8)) and all(t["end"] >= t["start"])
    assert all(t["tiles"][t["worked"] == 1] >= 1) and int(t["worked"].sum()) == 256
    for x in range(8):
        assert int(t["tiles"][t["xcc"] == x].sum()) == 32, x
    khz = asym.device_query(0)["wall_clock_khz"]
    mhz = t["cycles"].astype(np.float64) * khz / np.maximum(1, (t["end"] - t["start"]).astype(np.int64)) / 1e3
    assert np.all((mhz > 300) & (mhz < 2600)), (mhz.min(), mhz.max())  # the shader clock's range
    C.zero_()
    t = asym.gemm_trace(Ad, Bd, C, topo=topo, xcd_mask=0x0F)
    assert torch.equal(C, ref)
    assert int(t["tiles"].sum()) == 256 and set(t["xcc"][t["worked"] == 1].tolist()) <= {0, 1, 2, 3}
    span = (int(t["end"].max()) - int(t["start"].min())) / (khz / 1e3)
    print(f"traced 4096x4096x1024 on XCDs 0-3: {span:.1f} us from the first start to the last end")
    ts = asym.gemm_trace(Ad, Bd, C, topo=topo, launches=3)
    assert len(ts) == 3 and torch.equal(C, ref)
    for a, b in zip(ts, ts[1:]):  # queued on one stream: a launch starts after the previous one ends
        assert int(b["start"].min()) >= int(a["end"].max())
    # the small-M kernel has no traced form: a 32-row product is traced on the
    # persistent kernel and gives that kernel's bits
    C32 = torch.empty((32, 4096), dtype=torch.bfloat16, device=dev)
    t = asym.gemm_trace(Ad[:32], Bd, C32, topo=topo)
    prev = asym.set_small_m(False)
    try:
        ref32 = asym.gemm(Ad[:32], Bd, topo=topo)
    finally:
        asym.set_small_m(prev)
    torch.cuda.synchronize()
    assert torch.equal(C32, ref32) and int(t["tiles"].sum()) == t["plan"]["tiles_m"] * t["plan"]["tiles_n"]
    assert t["plan"]["small_m"] == 0
