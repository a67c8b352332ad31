"""GPU parity of the small-M kernel (at most 64 rows per row tile) against the
CPU oracle, through the C ABI.

Element by element over row counts on both sides of every 16-row block
boundary, ragged column counts (tiles with waves past N), K not a multiple of
the 32-wide k-step and K spanning one, two, three or many stages;
the decode projection 32 x 14336 x 4096 on sampled columns; bitwise: every
mapping, repeats and a CU-masked stream give the same bits, and on exact-integer
inputs the small-M kernel and the persistent kernel (the path switched off)
agree bit for bit with each other and with the integer product.  The plan says
which kernel a shape takes.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_24270_amd as asym
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


@pytest.mark.parametrize("M", [1, 5, 16, 17, 31, 32, 33, 48, 63, 64, 65, 100, 128, 200, 256])
@pytest.mark.parametrize("N,K", [(1000, 72), (96, 1000), (257, 4104), (40, 264), (1001, 72)])  # <= 2 row-tile WGs per CU
def test_small_m_elementwise(dev, M, N, K):
    p = workloads.make_problem(M, N, K, seed=100 + M)
    A, B = workloads.make_inputs(p)
    plan = asym.gemm_plan(A=A.to(dev), B=B.to(dev))
    assert plan["small_m"] == 1 and plan["tile_m"] == (16 if M <= 16 else 32 if M <= 32 else 64)
    assert plan["tiles_m"] == (M + plan["tile_m"] - 1) // plan["tile_m"]
    C = asym.gemm(A.to(dev), B.to(dev))
    torch.cuda.synchronize()
    R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
    err = assert_gemm_close(bits(C), R, what=f"{M}x{N}x{K}")
    assert err < 5e-3


def test_plan_picks_the_kernel(dev):
    def plan(M, K=4096, **kw):
        A = torch.zeros((M, K), dtype=torch.bfloat16, device=dev)
        B = torch.zeros((512, K), dtype=torch.bfloat16, device=dev)
        return asym.gemm_plan(A=A, B=B, **kw)
    assert plan(64)["small_m"] == 1 and plan(256)["small_m"] == 1 and plan(257)["small_m"] == 0
    # more than two 64-row workgroups per CU: the persistent kernel
    A = torch.zeros((256, 4096), dtype=torch.bfloat16, device=dev)
    B = torch.zeros((14336, 4096), dtype=torch.bfloat16, device=dev)
    assert asym.gemm_plan(A=A, B=B)["small_m"] == 0 and asym.gemm_plan(A=A[:128], B=B)["small_m"] == 1
    p65 = plan(65)
    # two 64-row tiles of 512 columns: 8-column tiles (64 x 2 workgroups, every CU
    # reading at most 8 columns of B; the aware grid pads 64 to a multiple of 8)
    assert (p65["tile_m"], p65["tiles_m"], p65["tile_n"], p65["grid"]) == (64, 2, 8, 128)
    assert plan(65, mapping="oblivious_rowmajor")["grid"] == 128
    assert plan(32, K=4100)["small_m"] == 0                       # K not a multiple of 8
    assert plan(32, xcd_mask=0x0F)["small_m"] == 0                # whole-XCD restriction
    p = plan(32)
    # 8 column tiles on 256 CUs: K split into 8 ranges (128 k-steps, at least 16 per range)
    assert (p["tile_n"], p["tiles_n"], p["k_splits"], p["grid"], p["claims"]) == (64, 8, 8, 64, 0)
    assert plan(32, K=256)["k_splits"] == 1 and plan(65)["k_splits"] == 1
    assert plan(200, mapping="aware")["grid"] == 256 and plan(200, mapping="oblivious_grouped")["grid"] == 256
    prev = asym.set_small_m(False)
    try:
        assert plan(32)["small_m"] == 0
    finally:
        asym.set_small_m(prev)


def test_decode_projection_sampled_and_bitwise(dev):
    (_, _), (da, db) = workloads.make_pd_inputs()
    A, B = da.to(dev), db.to(dev)
    outs = []
    for m in MAPS:
        for _ in range(2):
            outs.append(bits(asym.gemm(A, B, mapping=m)))
    assert all(np.array_equal(outs[0], o) for o in outs[1:])
    g = np.random.default_rng(3)
    cols = np.unique(np.concatenate([g.choice(14336, 512, replace=False), [14335]]))
    R, _ = oracle.gemm_bf16(bits(da), bits(db)[cols], "nk")
    err = assert_gemm_close(outs[0][:, cols], R, what="decode 32x14336x4096")
    print(f"decode 32x14336x4096 sampled max rel err {err:.3e}")


def test_exact_integer_small_equals_persistent(dev):
    p = workloads.make_problem(40, 3000, 2048, seed=7, dist="int")
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    small = bits(asym.gemm(Ad, Bd))
    prev = asym.set_small_m(False)
    try:
        pers = bits(asym.gemm(Ad, Bd))
    finally:
        asym.set_small_m(prev)
    _, Co = oracle.gemm_bf16(bits(A), bits(B), "nk")
    assert np.array_equal(small, Co) and np.array_equal(pers, Co)


def test_strided_operands(dev):
    M, N, K = 24, 700, 512
    p = workloads.make_problem(M, N, K, seed=9)
    A, B = workloads.make_inputs(p)
    Abig = torch.zeros((M, K + 64), dtype=torch.bfloat16)
    Abig[:, :K] = A
    Bbig = torch.zeros((N, K + 128), dtype=torch.bfloat16)
    Bbig[:, :K] = B
    Cbig = torch.full((M, N + 36), 7.0, dtype=torch.bfloat16, device=dev)
    Ad, Bd = Abig.to(dev)[:, :K], Bbig.to(dev)[:, :K]
    C = Cbig[:, :N]
    assert asym.gemm_plan(A=Ad, B=Bd, C=C)["small_m"] == 1
    asym.gemm(Ad, Bd, C)
    torch.cuda.synchronize()
    R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
    assert_gemm_close(bits(C), R)
    assert (Cbig[:, N:] == 7.0).all()   # columns past N untouched


def test_cu_masked_stream_bitwise(dev):
    topo = asym.probe_topology(0, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP)
    mask = workloads.random_mask_bits(11, 1, 128)[0]
    p = workloads.make_problem(32, 5000, 4096, seed=12, dist="llm")
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    ref = bits(asym.gemm(Ad, Bd))
    s = asym.stream_create(topo, mask)
    try:
        assert asym.gemm_plan(A=Ad, B=Bd, topo=topo, stream=s)["small_m"] == 1
        C = asym.gemm(Ad, Bd, topo=topo, stream=s)
        s.synchronize()
        assert np.array_equal(bits(C), ref)
    finally:
        asym.stream_destroy(s)


def test_grouped_small_groups_exact_integer_equals_persistent(dev):
    p = workloads.grouped_problem(32, 20, 4096, 2048, seed=5, dist="int")
    Ms, A, B = workloads.make_grouped_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    small = bits(asym.gemm_grouped(Ad, Bd, Ms))
    prev = asym.set_small_m(False)
    try:
        pers = bits(asym.gemm_grouped(Ad, Bd, Ms))
    finally:
        asym.set_small_m(prev)
    assert np.array_equal(small, pers)
    rows = np.cumsum([0] + Ms)
    for g in (0, 7, 31):
        _, Co = oracle.grouped_gemm_bf16(bits(A)[rows[g]:rows[g + 1]], bits(B)[g:g + 1], [Ms[g]], False)
        assert np.array_equal(small[rows[g]:rows[g + 1]], Co)


@pytest.mark.parametrize("M,N", [(200, 3000), (128, 14336), (130, 1000)])
def test_row_tiles_every_order_bitwise(dev, M, N):
    """Several 64-row tiles: the three placement orders give the same bits."""
    p = workloads.make_problem(M, N, 4096, seed=M, dist="llm")
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    outs = [bits(asym.gemm(Ad, Bd, mapping=m)) for m in MAPS]
    assert all(np.array_equal(outs[0], o) for o in outs[1:])
    g = np.random.default_rng(M)
    cols = np.unique(np.concatenate([g.choice(N, 256, replace=False), [N - 1]]))
    R, _ = oracle.gemm_bf16(bits(A), bits(B)[cols], "nk")
    assert_gemm_close(outs[0][:, cols], R, what=f"{M}x{N}x4096")


def test_grouped_groups_up_to_256_rows(dev):
    """Groups of 134..249 rows (the (32, 192) expert configuration's draw, 8
    groups kept): element by element against the oracle, bitwise across the
    orders, and bitwise equal to the persistent kernel on exact integers."""
    p = workloads.grouped_problem(8, 192, 1000, 512, seed=5)
    Ms, A, B = workloads.make_grouped_inputs(p)
    assert max(Ms) > 64 and max(Ms) <= 256
    Ad, Bd = A.to(dev), B.to(dev)
    outs = [bits(asym.gemm_grouped(Ad, Bd, Ms, mapping=m)) for m in MAPS]
    assert all(np.array_equal(outs[0], o) for o in outs[1:])
    R, _ = oracle.grouped_gemm_bf16(bits(A), bits(B), Ms)
    assert_gemm_close(outs[0], R, what="grouped up to 256 rows")
    pi = workloads.grouped_problem(8, 192, 1000, 512, seed=5, dist="int")
    Ms, A, B = workloads.make_grouped_inputs(pi)
    Ad, Bd = A.to(dev), B.to(dev)
    small = bits(asym.gemm_grouped(Ad, Bd, Ms))
    prev = asym.set_small_m(False)
    try:
        pers = bits(asym.gemm_grouped(Ad, Bd, Ms))
    finally:
        asym.set_small_m(prev)
    assert np.array_equal(small, pers)


@pytest.mark.parametrize("M,N,K", [(32, 4096, 4096), (16, 2000, 14336), (64, 1024, 8192), (5, 300, 1000)])
def test_split_k_elementwise_and_repeatable(dev, M, N, K):
    """Fewer column tiles than CUs: K is split across workgroups and a second
    launch adds the partial tiles in range order.  Element by element against
    the oracle; repeats and every mapping give the same bits."""
    p = workloads.make_problem(M, N, K, seed=M + N, dist="llm")
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    plan = asym.gemm_plan(A=Ad, B=Bd)
    assert plan["small_m"] == 1 and plan["k_splits"] > 1, plan
    outs = [bits(asym.gemm(Ad, Bd, mapping=m)) for m in MAPS for _ in range(2)]
    assert all(np.array_equal(outs[0], o) for o in outs[1:])
    R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
    err = assert_gemm_close(outs[0], R, what=f"split K {M}x{N}x{K}")
    print(f"{M}x{N}x{K}: {plan['k_splits']} K ranges, max rel err {err:.3e}")


def test_split_k_exact_integer_equals_persistent(dev):
    p = workloads.make_problem(32, 4096, 4096, seed=8, dist="int")
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    assert asym.gemm_plan(A=Ad, B=Bd)["k_splits"] > 1
    small = bits(asym.gemm(Ad, Bd))
    prev = asym.set_small_m(False)
    try:
        pers = bits(asym.gemm(Ad, Bd))
    finally:
        asym.set_small_m(prev)
    _, Co = oracle.gemm_bf16(bits(A), bits(B), "nk")
    assert np.array_equal(small, Co) and np.array_equal(pers, Co)


def test_split_k_under_an_xcd_restriction(dev):
    """32x4096x4096 splits K into ranges on the whole chip (small-M kernel);
    under a whole-XCD restriction it runs on the persistent kernel, one MFMA
    chain over K.  Both are within the tolerance of the oracle, and on
    exact-integer inputs (exact fp32 sums in any order) both equal it bitwise;
    on real-valued inputs the two may differ in the last bits, which the
    library documents."""
    for dist in ("llm", "int"):
        p = workloads.make_problem(32, 4096, 4096, seed=12, dist=dist)
        A, B = workloads.make_inputs(p)
        Ad, Bd = A.to(dev), B.to(dev)
        whole = asym.gemm_plan(A=Ad, B=Bd)
        restricted = asym.gemm_plan(A=Ad, B=Bd, xcd_mask=0xC0)
        assert whole["small_m"] == 1 and whole["k_splits"] == 8
        assert restricted["small_m"] == 0 and restricted["claims"] == 1
        C1 = bits(asym.gemm(Ad, Bd))
        C2 = bits(asym.gemm(Ad, Bd, xcd_mask=0xC0))
        torch.cuda.synchronize()
        R, Co = oracle.gemm_bf16(bits(A), bits(B), "nk")
        if dist == "int":
            assert np.array_equal(C1, Co) and np.array_equal(C2, Co)
        else:
            e1 = assert_gemm_close(C1, R, what="whole chip, K split")
            e2 = assert_gemm_close(C2, R, what="XCDs 6-7, persistent kernel")
            print(f"32x4096x4096: split {e1:.3e}, restricted {e2:.3e}, "
                  f"bitwise equal share {float(np.mean(C1 == C2)):.4f}")


@pytest.mark.parametrize("M,N,K,width", [(32, 14336, 4096, 56), (32, 10240, 4096, 40), (40, 3000, 200, 16),
                                         (128, 4096, 4096, 32), (128, 14336, 4096, 64), (100, 1000, 72, 8)])
def test_narrow_column_tiles(dev, M, N, K, width):
    """An unsplit product takes the column-tile width (a multiple of 8 up to
    64) that minimises the columns of B the busiest CU reads (a wave of 8
    columns or an idle one at the tile's edge; one or more row tiles).  On exact-integer inputs it
    equals the oracle and the persistent kernel bitwise; on real-valued ones
    every mapping gives the same bits and sampled columns match the oracle."""
    ncu = asym.device_query(0)["n_cus"]
    p = workloads.make_problem(M, N, K, seed=N + K, dist="int")
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    plan = asym.gemm_plan(A=Ad, B=Bd)
    assert plan["small_m"] == 1 and plan["k_splits"] == 1, plan
    if ncu == 256:
        assert plan["tile_n"] == width and plan["tiles_n"] == (N + width - 1) // width, plan
    small = bits(asym.gemm(Ad, Bd))
    prev = asym.set_small_m(False)
    try:
        pers = bits(asym.gemm(Ad, Bd))
    finally:
        asym.set_small_m(prev)
    _, Co = oracle.gemm_bf16(bits(A), bits(B), "nk")
    assert np.array_equal(small, Co) and np.array_equal(pers, Co)
    p = workloads.make_problem(M, N, K, seed=N + K + 1)
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    outs = [bits(asym.gemm(Ad, Bd, mapping=m)) for m in MAPS]
    assert all(np.array_equal(outs[0], o) for o in outs[1:])
    g = np.random.default_rng(N)
    cols = np.unique(np.concatenate([g.choice(N, min(N, 400), replace=False), np.arange(N - width, N)]))
    R, _ = oracle.gemm_bf16(bits(A), bits(B)[cols], "nk")
    assert_gemm_close(outs[0][:, cols], R, what=f"{M}x{N}x{K} in {width}-column tiles")
