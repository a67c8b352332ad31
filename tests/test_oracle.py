"""Pins for the CPU oracle GEMM against facts other than itself.

Each test checks the oracle against something the mathematics fixes:
exact rational arithmetic, exact integer products, algebraic invariants,
an fp64 library product within Higham's summation bound, a closed-form case
where only the k order decides the sum, and torch's bf16 rounding.
"""
from fractions import Fraction
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_24270_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
U = 2.0 ** -24  # unit roundoff of fp32


def bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def f32_of_bits(h: np.ndarray) -> np.ndarray:
    return oracle.bf16_bits_to_f32(h)


def gamma(k: int) -> float:
    return k * U / (1 - k * U)


def torch_rne(x_f32: np.ndarray) -> np.ndarray:
    return bits(torch.from_numpy(np.ascontiguousarray(x_f32, dtype=np.float32)).to(torch.bfloat16))


# -- bf16 rounding ---------------------------------------------------------

def test_bf16_golden_values():
    rows = []
    with open(os.path.join(GOLDEN, "bf16_rne.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                a, b = line.split()
                rows.append((int(a, 16), int(b, 16)))
    x = np.array([r[0] for r in rows], dtype=np.uint32).view(np.float32)
    got = oracle.f32_to_bf16(x)
    want = np.array([r[1] for r in rows], dtype=np.uint16)
    assert np.array_equal(got, want), list(zip(got, want))


def test_bf16_rne_matches_torch_on_2pow20_values():
    rng = np.random.default_rng(20)
    n = 1 << 20
    u = rng.integers(0, 2 ** 32, size=n, dtype=np.uint64).astype(np.uint32)
    # a quarter of them made exact ties (low 16 bits = 0x8000), both parities
    u[: n // 4] = (u[: n // 4] & 0xFFFF0000) | 0x8000
    # drop NaNs (their payload handling is not compared)
    x = u.view(np.float32)
    x = x[~np.isnan(x)]
    assert np.array_equal(oracle.f32_to_bf16(x), torch_rne(x))


# -- brute force in exact rationals ---------------------------------------

@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (2, 3, 5), (3, 5, 8), (5, 2, 17),
                                   (8, 17, 3), (17, 8, 2), (17, 17, 17)])
def test_brute_force_tiny(M, N, K):
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=100 + M * 31 + N * 7 + K))
    Ab, Bb = bits(A), bits(B)                       # A [M,K], B stored [N,K]
    R, C = oracle.gemm_bf16(Ab, Bb, "nk")
    a, b = f32_of_bits(Ab), f32_of_bits(Bb)
    for i in range(M):
        for j in range(N):
            exact = sum((Fraction(float(a[i, k])) * Fraction(float(b[j, k])) for k in range(K)),
                        Fraction(0))
            absum = sum(abs(float(a[i, k]) * float(b[j, k])) for k in range(K))
            assert abs(Fraction(float(R[i, j])) - exact) <= Fraction(gamma(K) * absum), (i, j)
    # the bf16 output is the library's RNE of the fp32 result
    assert np.array_equal(C, torch_rne(R))


def test_k_order_golden():
    with open(os.path.join(GOLDEN, "k_order.txt")) as f:
        vals = [line.split() for line in f if line.strip() and not line.startswith("#")]
    K = int(vals[0][0])
    a = np.array([float(v) for v in vals[1]], dtype=np.float32).reshape(1, K)
    b = np.array([float(v) for v in vals[2]], dtype=np.float32).reshape(1, K)  # [N=1, K]
    want_seq, want_exact = float(vals[3][0]), float(vals[4][0])
    R, _ = oracle.gemm_bf16(torch_rne(a), torch_rne(b), "nk")
    assert float(R[0, 0]) == want_seq
    assert float(np.dot(a.astype(np.float64)[0], b.astype(np.float64)[0])) == want_exact


# -- exact-integer regime ---------------------------------------------------

@pytest.mark.parametrize("M,N,K", [(64, 48, 1000), (33, 129, 257), (1, 7, 4099)])
def test_exact_integer_regime(M, N, K):
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=7, dist="int"))
    Ab, Bb = bits(A), bits(B)
    want = A.to(torch.int64).numpy() @ B.to(torch.int64).numpy().T
    for lay, Bl in (("nk", Bb), ("kn", np.ascontiguousarray(Bb.T))):
        R, C = oracle.gemm_bf16(Ab, Bl, lay)
        assert np.array_equal(R.astype(np.int64), want)
        assert np.array_equal(C, torch_rne(want.astype(np.float32)))


# -- invariants -------------------------------------------------------------

def test_identity_zero_transpose_layouts():
    M, N, K = 37, 53, 64
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=11))
    Ab, Bb = bits(A), bits(B)
    # A . I = A  (B stored [N=K, K] as the identity)
    I_nk = bits(torch.eye(K, dtype=torch.bfloat16))
    _, C = oracle.gemm_bf16(Ab, I_nk, "nk")
    assert np.array_equal(C, Ab)
    # I . B = B (logical B is the transpose of the stored [N,K] array)
    I_m = bits(torch.eye(K, dtype=torch.bfloat16))
    _, C = oracle.gemm_bf16(I_m, Bb, "nk")
    assert np.array_equal(C, Bb.T)
    # A . 0 = 0
    _, C = oracle.gemm_bf16(Ab, np.zeros_like(Bb), "nk")
    assert np.array_equal(f32_of_bits(C), np.zeros((M, N), np.float32))
    # (A . B)^T = B^T . A^T, bitwise: same products, same k order
    R1, C1 = oracle.gemm_bf16(Ab, Bb, "nk")
    R2, C2 = oracle.gemm_bf16(Bb, Ab, "nk")
    assert np.array_equal(R1.T, R2) and np.array_equal(C1.T, C2)
    # [N,K] and [K,N] storage of the same logical B agree bitwise
    R3, C3 = oracle.gemm_bf16(Ab, np.ascontiguousarray(Bb.T), "kn")
    assert np.array_equal(R1, R3) and np.array_equal(C1, C3)


def test_fp64_library_product_within_higham_bound():
    M = N = K = 256
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=3))
    Ab, Bb = bits(A), bits(B)
    R, _ = oracle.gemm_bf16(Ab, Bb, "nk")
    a, b = f32_of_bits(Ab).astype(np.float64), f32_of_bits(Bb).astype(np.float64)
    exact = a @ b.T
    bound = gamma(K) * (np.abs(a) @ np.abs(b).T)
    err = np.abs(R.astype(np.float64) - exact)
    assert np.all(err <= bound + 1e-300)
    # and the bound is not vacuous: the sum does round somewhere
    assert np.any(err > 0)


def test_rejects_bad_arguments():
    with pytest.raises(ValueError):
        oracle.gemm_bf16(np.zeros((2, 3), np.uint16), np.zeros((2, 4), np.uint16), "nk")
    with pytest.raises(ValueError):
        oracle.gemm_bf16(np.zeros((2, 3), np.uint16), np.zeros((3, 2), np.uint16), "xx")


def test_row_permutation_equivariant():
    M, N, K = 96, 80, 300
    A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=5))
    R1, C1 = oracle.gemm_bf16(bits(A), bits(B), "nk")
    # a permutation of output rows permutes the result rows exactly
    perm = np.random.default_rng(0).permutation(M)
    R2, C2 = oracle.gemm_bf16(bits(A)[perm], bits(B), "nk")
    assert np.array_equal(R1[perm], R2) and np.array_equal(C1[perm], C2)


# ---- grouped GEMM oracle ------------------------------------------------------

def _grouped_case(rows, N, K, seed, dist="uniform"):
    p = workloads.GroupedProblem("t", len(rows), 1, N, K, seed=seed, dist=dist)
    Ms, A, B = workloads.make_grouped_inputs(p, rows=rows)
    return Ms, bits(A), bits(B.reshape(len(rows) * N, K)).reshape(len(rows), N, K)


def test_grouped_one_group_is_the_plain_gemm():
    Ms, A, B = _grouped_case([77], 40, 130, seed=11)
    R, C = oracle.grouped_gemm_bf16(A, B, Ms)
    R1, C1 = oracle.gemm_bf16(A, B[0], "nk")
    assert np.array_equal(C, C1) and np.array_equal(R, R1)


def test_grouped_shared_weights_are_one_gemm_of_the_packed_rows():
    """With every group's weights equal, the grouped product of the packed rows
    is one plain product of all of them: row offsets and packing are pinned."""
    Ms, A, B = _grouped_case([5, 0, 33, 1, 17], 24, 72, seed=12)
    Bs = np.repeat(B[:1], len(Ms), axis=0)
    R, C = oracle.grouped_gemm_bf16(A, Bs, Ms)
    R1, C1 = oracle.gemm_bf16(A, B[0], "nk")
    assert np.array_equal(C, C1) and np.array_equal(R, R1)


def test_grouped_permuting_groups_permutes_row_blocks():
    """Reordering the groups (rows and weights together) reorders the output
    blocks and changes nothing else: each group meets its own weights."""
    Ms, A, B = _grouped_case([9, 4, 0, 21, 13], 16, 96, seed=13)
    R, C = oracle.grouped_gemm_bf16(A, B, Ms)
    starts = np.cumsum([0] + Ms)
    perm = [3, 0, 4, 2, 1]
    A2 = np.concatenate([A[starts[g]:starts[g + 1]] for g in perm])
    C_expect = np.concatenate([C[starts[g]:starts[g + 1]] for g in perm])
    R2, C2 = oracle.grouped_gemm_bf16(A2, B[perm], [Ms[g] for g in perm])
    assert np.array_equal(C2, C_expect)
    # and the weights matter: pairing every group with group 0's weights differs
    _, C3 = oracle.grouped_gemm_bf16(A, np.repeat(B[:1], len(Ms), axis=0), Ms)
    assert not np.array_equal(C3, C)


def test_grouped_exact_integer_closed_form():
    """Integer inputs: every product and partial sum is exact, so each group's
    block equals the integer product, converted once."""
    Ms, A, B = _grouped_case([3, 7, 2], 12, 40, seed=14, dist="int")
    R, C = oracle.grouped_gemm_bf16(A, B, Ms)
    Af = oracle.bf16_bits_to_f32(A).astype(np.int64)
    Bf = oracle.bf16_bits_to_f32(B).astype(np.int64)
    row = 0
    for g, m in enumerate(Ms):
        exact = Af[row:row + m] @ Bf[g].T
        assert np.array_equal(R[row:row + m], exact.astype(np.float32))
        row += m


def test_grouped_row_sampling_follows_the_definition():
    """M_i = floor(M U_i), U_i in [0.7, 1.3): every count within the range,
    reproducible from the seed."""
    for G, M in workloads.GROUPED_GM:
        p = workloads.grouped_problem(G, M, 64, 64)
        rows = p.rows()
        assert len(rows) == G and rows == p.rows()
        assert all(int(0.7 * M) <= r <= int(1.3 * M) for r in rows)
    p = workloads.GROUPED[0]
    assert p.working_set_bytes == 2 * (sum(p.rows()) * (p.K + p.N) + p.G * p.N * p.K)
