"""The GEMM entry point that allocates nothing (asym_gemm_bf16_noalloc),
called through the C ABI and compared with asym_gemm_bf16, which runs the same
kernels with its per-stream workspace: the results must be bitwise equal.
Calls come in a row, each next one smaller or of another kind, so that what
the shared per-GPU array holds from the call before (a larger schedule, other
partials, used counters) is exercised: the persistent kernel's static aware
form, the claiming form (whole-XCD restriction, uneven CU set), the oblivious
orders, and the small-M kernel with a split K.
"""
import numpy as np
import pytest
import torch

import oracle
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


# (M, N, K, distribution, mapping, xcd_mask), run in this order
SEQUENCE = [
    (2048, 2048, 1024, "uniform", "aware", 0),          # static aware, 64 tiles
    (512, 768, 256, "uniform", "aware", 0),             # smaller: 2 x 3 tiles
    (1024, 1536, 512, "llm", "aware", 0x0F),            # claiming form, counters used
    (300, 520, 264, "uniform", "aware", 0x0F),          # again, smaller (counters reused)
    (32, 6144, 4096, "llm", "aware", 0),                # small-M decode projection, K in 8 ranges
    (32, 4096, 4096, "llm", "aware", 0),                # small-M, K split into 8 ranges
    (24, 600, 2048, "llm", "aware", 0),                 # small-M, smaller split
    (700, 900, 640, "uniform", "oblivious_grouped", 0),  # oblivious orders
    (640, 512, 128, "uniform", "oblivious_rowmajor", 0),
    (200, 136, 150, "uniform", "aware", 0),             # predicated path (K not a multiple of 8)
]


def test_noalloc_equals_the_workspace_entry_point(dev, topo):
    lim = asym.noalloc_limits()
    print("limits", lim)
    assert lim["scratch_bytes"] <= 32 << 20 and lim["max_tiles"] > 200000
    for i, (M, N, K, dist, mapping, xm) in enumerate(SEQUENCE):
        print(f"case {i}: {M}x{N}x{K} {dist} {mapping} xcd_mask={xm:#x}", flush=True)
        A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=40 + i, dist=dist))
        Ad, Bd = A.to(dev), B.to(dev)
        ref = asym.gemm(Ad, Bd, mapping=mapping, topo=topo, xcd_mask=xm)
        C = torch.full_like(ref, 3.0)
        asym.gemm_noalloc(Ad, Bd, C, topo, mapping=mapping, xcd_mask=xm)
        torch.cuda.synchronize()
        assert torch.equal(C, ref), i
        if i in (1, 6, 9):
            R, _ = oracle.gemm_bf16(bits(A), bits(B), "nk")
            assert_gemm_close(bits(C), R, what=f"no-alloc case {i}")


def test_noalloc_on_an_uneven_cu_set(dev, topo):
    """A seeded random 128-CU set (unequal per-XCD counts): the claiming form
    on a masked stream, twice in a row with a smaller second problem."""
    mask = workloads.random_mask_bits(4, 1, 128)[0]
    s = asym.stream_create(topo, mask)
    try:
        for i, (M, N, K) in enumerate(((1536, 2048, 768), (512, 640, 384))):
            A, B = workloads.make_inputs(workloads.make_problem(M, N, K, seed=70 + i))
            Ad, Bd = A.to(dev), B.to(dev)
            torch.cuda.synchronize()
            assert asym.gemm_plan(A=Ad, B=Bd, topo=topo, stream=s)["claims"] == 1
            ref = asym.gemm(Ad, Bd, topo=topo, stream=s)
            C = torch.zeros_like(ref)
            s.synchronize()
            asym.gemm_noalloc(Ad, Bd, C, topo, stream=s)
            s.synchronize()
            assert torch.equal(C, ref), i
    finally:
        asym.stream_destroy(s)


def test_noalloc_rejects_what_it_cannot_serve(dev, topo):
    A = torch.zeros((64, 64), dtype=torch.bfloat16, device=dev)
    C = torch.zeros((64, 64), dtype=torch.bfloat16, device=dev)
    lib = asym.load_library()
    import ctypes
    pa, pc = ctypes.c_void_p(A.data_ptr()), ctypes.c_void_p(C.data_ptr())
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    # no topology: refused (a first-use probe would allocate)
    assert lib.asym_gemm_bf16_noalloc(None, 64, 64, 64, pa, 64, pa, 64, asym.B_NK, pc, 64, 0, 0, s) == asym.EINVAL
    # B stored [K][N]: refused (it would need a transposed copy of B)
    assert lib.asym_gemm_bf16_noalloc(topo.handle, 64, 64, 64, pa, 64, pa, 64, asym.B_KN, pc, 64, 0, 0, s) == \
        asym.EUNSUPPORTED
    torch.cuda.synchronize()
