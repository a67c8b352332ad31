"""The benchmark's own parity check: the CPU-baseline leg times the oracle and,
given the GPU's output of the timed problem, compares every element with the
oracle's fp32 sum before rounding (gate max |C - R32| / max(|R32|, rms) <= 2e-2).
Here the "GPU output" is built on the CPU, so the check itself is exercised
without a GPU: a correctly rounded product passes, a planted 10% error in one
element fails."""
import os
import sys

import torch

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _inputs(seed=3, M=96, N=80, K=136):
    g = torch.Generator().manual_seed(seed)
    A = (torch.rand(M, K, generator=g) * 2 - 1).to(torch.bfloat16)
    B = (torch.rand(N, K, generator=g) * 2 - 1).to(torch.bfloat16)
    return A, B


def test_correct_output_passes():
    A, B = _inputs()
    C = (A.double() @ B.double().t()).to(torch.bfloat16)  # rounded from the exact product
    cpu, par = bench.cpu_baseline(A, B, A.shape[0], C)
    assert cpu["kind"] == "oracle" and cpu["value"] > 0
    assert par["pass"] and par["max_rel_err"] <= 2.0 ** -8
    assert par["bitwise_equal_to_oracle_frac"] > 0.99


def test_planted_error_fails():
    A, B = _inputs()
    C = (A.double() @ B.double().t()).to(torch.bfloat16)
    C[7, 11] = C[7, 11] * 1.1 + 0.5
    _, par = bench.cpu_baseline(A, B, A.shape[0], C)
    assert not par["pass"] and par["max_rel_err"] > 2e-2


def test_rows_subset_checks_only_those_rows():
    A, B = _inputs()
    C = (A.double() @ B.double().t()).to(torch.bfloat16)
    C[-1, 0] = -C[-1, 0] * 3 + 1  # outside the checked rows
    cpu, par = bench.cpu_baseline(A, B, 32, C)
    assert par["pass"] and "rows 0..31" in par["checked"]


def test_no_gpu_output_times_only():
    A, B = _inputs()
    cpu, par = bench.cpu_baseline(A, B, 16)
    assert par is None and cpu["unit"] == "TFLOP/s"
