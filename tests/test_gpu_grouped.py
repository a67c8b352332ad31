"""GPU parity of the grouped GEMM (the mixture-of-experts expert layer) against
the CPU oracle, through the C ABI.

Small ragged cases are compared element by element, including empty groups,
one-row groups and groups that end inside a tile; a full configuration of the
paper's small-M kind is compared element by element too, and a large-M one on
sampled rows of every group.  Exact-integer inputs must give the oracle's bits;
every mapping and CU set gives the same bits.
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


def bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    asym.load_library()
    torch.cuda.set_device(0)
    return torch.device("cuda:0")


def inputs(rows, N, K, seed, dist="uniform"):
    p = workloads.GroupedProblem("t", len(rows), 1, N, K, seed=seed, dist=dist)
    return workloads.make_grouped_inputs(p, rows=rows)


def run(A, B, Ms, mapping="aware", **kw):
    C = asym.gemm_grouped(A, B, Ms, mapping=mapping, **kw)
    torch.cuda.synchronize()
    return C


@pytest.mark.parametrize("rows,N,K", [([0, 300, 17, 256, 1], 520, 264), ([1, 2, 3], 700, 328),
                                      ([513, 0, 0, 40], 192, 64), ([7], 1031, 200)])
def test_grouped_small_elementwise(dev, rows, N, K):
    Ms, A, B = inputs(rows, N, K, seed=len(rows) + N)
    ref, _ = oracle.grouped_gemm_bf16(bits(A), bits(B), Ms)
    Ad, Bd = A.to(dev), B.to(dev)
    C = run(Ad, Bd, Ms)
    e = assert_gemm_close(bits(C), ref, what=f"grouped {rows} x {N} x {K}")
    print(f"grouped {rows} N={N} K={K}: max rel err {e:.3e}")
    for m in MAPS[1:]:
        assert torch.equal(run(Ad, Bd, Ms, m), C), m


def test_grouped_unaligned_k_takes_the_predicated_path(dev):
    Ms, A, B = inputs([33, 0, 290], 136, 150, seed=3)
    ref, _ = oracle.grouped_gemm_bf16(bits(A), bits(B), Ms)
    assert_gemm_close(bits(run(A.to(dev), B.to(dev), Ms)), ref, what="grouped K=150")


def test_grouped_paper_small_m_config_elementwise(dev):
    """(G, M) = (32, 20) with (N, K) = (4096, 4096): every output element."""
    p = workloads.grouped_problem(32, 20, 4096, 4096)
    Ms, A, B = workloads.make_grouped_inputs(p)
    ref, _ = oracle.grouped_gemm_bf16(bits(A), bits(B), Ms)
    Ad, Bd = A.to(dev), B.to(dev)
    C = run(Ad, Bd, Ms)
    e = assert_gemm_close(bits(C), ref, what=p.name)
    print(f"{p.name} rows {sum(Ms)}: max rel err {e:.3e}")
    assert torch.equal(run(Ad, Bd, Ms, "oblivious_grouped"), C)


def test_grouped_paper_large_m_exact_integer_sampled(dev):
    """(G, M) = (6, 1024) with (N, K) = (4096, 2048), integer inputs: sampled
    rows of every group (first, last, random) give the oracle's bits."""
    p = workloads.grouped_problem(6, 1024, 4096, 2048, dist="int")
    Ms, A, B = workloads.make_grouped_inputs(p)
    C = run(A.to(dev), B.to(dev), Ms)
    Cb, Ab, Bb = bits(C), bits(A), bits(B)
    g = np.random.default_rng(0)
    row = 0
    for i, m in enumerate(Ms):
        pick = np.unique(np.concatenate([[0, m - 1], g.choice(m, size=min(14, m), replace=False)]))
        _, ref = oracle.gemm_bf16(Ab[row + pick], Bb[i], "nk")
        assert np.array_equal(Cb[row + pick], ref), f"group {i}"
        row += m


def test_grouped_uneven_cu_set_is_bitwise_the_same(dev):
    """On a random 128-CU set (unequal XCD counts: the claiming form) the
    grouped GEMM gives the full chip's bits."""
    topo = asym.probe_topology(0, asym.PROBE_IDENTITY | asym.PROBE_MASKMAP)
    Ms, A, B = inputs([300, 20, 0, 700, 64, 5], 1024, 512, seed=21)
    Ad, Bd = A.to(dev), B.to(dev)
    ref = run(Ad, Bd, Ms)
    mask = workloads.random_mask_bits(7, 1, 128)[0]
    s = asym.stream_create(topo, mask)
    try:
        for m in MAPS:
            C = asym.gemm_grouped(Ad, Bd, Ms, mapping=m, topo=topo, stream=s)
            s.synchronize()
            assert torch.equal(C, ref), m
    finally:
        asym.stream_destroy(s)


def test_grouped_all_empty_is_a_no_op(dev):
    B = torch.zeros((3, 64, 32), dtype=torch.bfloat16, device=dev)
    A = torch.zeros((0, 32), dtype=torch.bfloat16, device=dev)
    C = run(A, B, [0, 0, 0])
    assert tuple(C.shape) == (0, 64)


def test_grouped_rejects_bad_arguments(dev):
    B = torch.zeros((2, 64, 32), dtype=torch.bfloat16, device=dev)
    A = torch.zeros((5, 32), dtype=torch.bfloat16, device=dev)
    with pytest.raises(asym.AsymError) as e:
        asym.gemm_grouped(A, B, [6, -1])
    assert e.value.status == asym.EINVAL
    with pytest.raises(ValueError):
        asym.gemm_grouped(A, B, [2, 2])   # A has 5 rows, not 4


def test_grouped_tables_reused_and_evicted(dev):
    """Ten different row splits of the same rows (more than the library keeps
    tables for), each run three times interleaved: repeated calls reuse their
    tables or rebuild them after eviction, always with the same bits, and
    spot checks against the oracle hold."""
    rng = np.random.default_rng(5)
    splits = []
    for _ in range(10):
        cuts = np.sort(rng.choice(np.arange(1, 600), size=3, replace=False))
        splits.append([int(x) for x in np.diff(np.concatenate([[0], cuts, [600]]))])
    Ms0, A, B = inputs([150, 150, 150, 150], 384, 256, seed=31)
    Ad, Bd = A.to(dev), B.to(dev)
    first = {}
    for rep in range(3):
        for i, Ms in enumerate(splits):
            C = run(Ad, Bd, Ms, mapping=MAPS[(i + rep) % 3])
            if rep == 0:
                first[i] = C.clone()
            else:
                assert torch.equal(C, first[i]), (rep, i)
    for i in (0, 7):
        ref, _ = oracle.grouped_gemm_bf16(bits(A), bits(B), splits[i])
        assert_gemm_close(bits(first[i]), ref, what=f"split {splits[i]}")
