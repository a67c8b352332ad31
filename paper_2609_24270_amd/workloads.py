"""Seeded synthetic workloads shared by the tests, the benchmark and the oracle.

This module only draws inputs: it holds none of the method's arithmetic (no
product, no rounding beyond torch's own fp32->bf16 conversion of the draws, no
scheduling), so the HIP path and the CPU oracle can both consume its output
without sharing code.

Recipe (one torch CPU generator per GEMM problem, seeded as listed):
  * A is drawn first, then B, each in fp32 in its storage shape and converted
    to bf16 with torch's round-to-nearest-even;
  * uniform[-1,1]: torch.rand(...) * 2 - 1;  normal(0, s): torch.randn(...) * s;
  * B is stored [N, K] (the K-contiguous weight layout); a [K, N] copy is the
    transpose of the same logical matrix.
The shapes are those of the paper's workload classes transplanted to a bf16
GEMM: square GEMMs, and the three projection shapes of an 8B-class decoder
layer (hidden 4096, FFN 14336, fused QKV 6144) with 4096 tokens.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class GemmProblem:
    name: str
    M: int
    N: int
    K: int
    seed: int
    dist: str = "uniform"      # "uniform" | "llm" | "int"
    a_sigma: float = 1.0       # llm: activation std
    b_sigma: float = 0.02      # llm: weight std

    @property
    def flops(self) -> float:
        return 2.0 * self.M * self.N * self.K


# Square GEMM, 512^3, the small parity case (the oracle finishes in seconds).
SQUARE_512 = GemmProblem("square_512", 512, 512, 512, seed=0)
# Square GEMM, 8192^3, the headline full-GPU case.
SQUARE_8192 = GemmProblem("square_8192", 8192, 8192, 8192, seed=1)
# 8B-class decoder projections at 4096 tokens (FFN up, FFN down, fused QKV).
LLM_SHAPES = (
    GemmProblem("llm_ffn_up", 4096, 14336, 4096, seed=2, dist="llm"),
    GemmProblem("llm_ffn_down", 4096, 4096, 14336, seed=2, dist="llm"),
    GemmProblem("llm_qkv", 4096, 6144, 4096, seed=2, dist="llm"),
)
# Prefill / decode GEMMs multiplexed on two CU partitions (seed 3, one generator:
# prefill A, B then decode A, B).
PREFILL = GemmProblem("prefill", 8192, 4096, 4096, seed=3, dist="llm")
DECODE = GemmProblem("decode", 32, 14336, 4096, seed=3, dist="llm")
# Co-location sweep GEMM (seed 4), uniform inputs.
COLOC = GemmProblem("coloc_4096", 4096, 4096, 4096, seed=4)
COPY_BYTES = 64 << 20


def _draw(g: torch.Generator, shape, dist: str, sigma: float) -> torch.Tensor:
    if dist == "uniform":
        x = torch.rand(shape, generator=g, dtype=torch.float32) * 2.0 - 1.0
    elif dist == "normal":
        x = torch.randn(shape, generator=g, dtype=torch.float32) * sigma
    elif dist == "int":
        # integers in {-2,...,2}: every partial sum of a K <= 2^20 dot product
        # is an integer below 2^24, so fp32 accumulation is exact in any order
        x = torch.randint(-2, 3, shape, generator=g).to(torch.float32)
    else:
        raise ValueError(dist)
    return x.to(torch.bfloat16)


def make_inputs_from(g: torch.Generator, p: GemmProblem):
    """Draw (A [M,K], B [N,K]) bf16 CPU tensors for problem p from generator g."""
    if p.dist == "llm":
        A = _draw(g, (p.M, p.K), "normal", p.a_sigma)
        B = _draw(g, (p.N, p.K), "normal", p.b_sigma)
    else:
        A = _draw(g, (p.M, p.K), p.dist, 1.0)
        B = _draw(g, (p.N, p.K), p.dist, 1.0)
    return A, B


def make_inputs(p: GemmProblem):
    """(A [M,K], B [N,K]) bf16 CPU tensors for p from a fresh generator."""
    g = torch.Generator(device="cpu").manual_seed(p.seed)
    return make_inputs_from(g, p)


def make_pd_inputs():
    """Prefill then decode inputs from one generator seeded 3."""
    g = torch.Generator(device="cpu").manual_seed(PREFILL.seed)
    pa, pb = make_inputs_from(g, PREFILL)
    da, db = make_inputs_from(g, DECODE)
    return (pa, pb), (da, db)


def make_problem(M: int, N: int, K: int, seed: int, dist: str = "uniform") -> GemmProblem:
    return GemmProblem(f"gemm_{M}x{N}x{K}", M, N, K, seed=seed, dist=dist)


# Grouped GEMM, the mixture-of-experts expert layer (Section 7.1 and its
# appendix): G groups with expected row count M; group i has
# M_i = floor(M * U_i) rows, U_i ~ Uniform(0.7, 1.3), drawn per shape seed.
# The configurations are every (G, M) in GROUPED_GM with every (N, K) in
# GROUPED_NK.  Recipe: one torch CPU generator per problem, seeded with
# `seed`; the G values U_i are drawn first (float64), then A [sum M_i, K] ~
# normal(0, 1) and B [G, N, K] ~ normal(0, 0.02), converted to bf16.
GROUPED_GM = ((32, 192), (6, 1024), (32, 20), (6, 20))
GROUPED_NK = ((6144, 7168), (7168, 3072), (4096, 4096), (4096, 2048))


@dataclass(frozen=True)
class GroupedProblem:
    name: str
    G: int
    M: int          # expected rows per group
    N: int
    K: int
    seed: int
    dist: str = "llm"    # "llm" | "uniform" | "int"

    def rows(self):
        g = torch.Generator(device="cpu").manual_seed(self.seed)
        return _group_rows(g, self.G, self.M)

    @property
    def flops(self) -> float:
        return 2.0 * sum(self.rows()) * self.N * self.K

    @property
    def working_set_bytes(self) -> int:
        """Logical bytes of inputs and output: 2 (sum M_i (K + N) + G N K)."""
        return 2 * (sum(self.rows()) * (self.K + self.N) + self.G * self.N * self.K)


def _group_rows(g: torch.Generator, G: int, M: int):
    u = torch.rand(G, generator=g, dtype=torch.float64) * 0.6 + 0.7
    return [int(math.floor(M * float(x))) for x in u]


def grouped_problem(G: int, M: int, N: int, K: int, seed: int = 5, dist: str = "llm") -> GroupedProblem:
    return GroupedProblem(f"group_G{G}_M{M}_N{N}_K{K}_s{seed}", G, M, N, K, seed=seed, dist=dist)


GROUPED = tuple(grouped_problem(G, M, N, K) for (G, M) in GROUPED_GM for (N, K) in GROUPED_NK)


def make_grouped_inputs(p: GroupedProblem, rows=None):
    """(row counts, A [sum M_i, K], B [G, N, K]) bf16 CPU tensors for p.  `rows`
    overrides the sampled row counts (the generator still draws them first)."""
    g = torch.Generator(device="cpu").manual_seed(p.seed)
    Ms = _group_rows(g, p.G, p.M)
    if rows is not None:
        Ms = list(rows)
    total = sum(Ms)
    if p.dist == "llm":
        A = _draw(g, (total, p.K), "normal", 1.0)
        B = _draw(g, (p.G, p.N, p.K), "normal", 0.02)
    else:
        A = _draw(g, (total, p.K), p.dist, 1.0)
        B = _draw(g, (p.G, p.N, p.K), p.dist, 1.0)
    return Ms, A, B


def make_grouped_inputs_on(p: GroupedProblem, device):
    """(row counts, A, B) like make_grouped_inputs, with A and B drawn on
    `device` by a generator there seeded with p.seed (same distributions,
    different streams of numbers; for timing runs at the full sizes, where
    drawing gigabytes on the CPU would take minutes).  The row counts are the
    CPU draw, identical to make_grouped_inputs."""
    Ms = p.rows()
    g = torch.Generator(device=device).manual_seed(p.seed)
    if p.dist != "llm":
        raise ValueError("device draws support the llm recipe only")
    A = torch.randn((sum(Ms), p.K), generator=g, device=device).to(torch.bfloat16)
    B = torch.empty((p.G, p.N, p.K), dtype=torch.bfloat16, device=device)
    for i in range(p.G):  # one group at a time keeps the fp32 draw small
        B[i] = (torch.randn((p.N, p.K), generator=g, device=device) * 0.02).to(torch.bfloat16)
    return Ms, A, B


def random_mask_bits(seed: int, n_masks: int, n_bits: int, total: int = 256):
    """n_masks seeded random subsets of n_bits CU-mask bit positions out of total.

    Each subset is the first n_bits entries of a seeded permutation, drawn the
    way a topology-oblivious user would pick CUs: over mask bits, by count.
    """
    g = torch.Generator(device="cpu").manual_seed(seed)
    out = []
    for _ in range(n_masks):
        perm = torch.randperm(total, generator=g)
        out.append(sorted(int(b) for b in perm[:n_bits]))
    return out


def copy_source(n_elems: int, seed: int = COLOC.seed + 1000) -> torch.Tensor:
    """Arbitrary bf16 bit patterns (finite) for the streaming-copy source."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    return (torch.rand(n_elems, generator=g) * 2 - 1).to(torch.bfloat16)


# Synthetic per-address latencies with a planted affinity structure, input to
# the affinity analysis in host-only tests.  XCD x belongs to group grp[x];
# each address gets a uniformly drawn home group h; its latency from x is
# tier[dist[grp[x]][h]] plus a per-address offset shared by all XCDs (uniform in
# [0, common)) plus per-(XCD, address) jitter (uniform in [0, jitter)).
# Appendix G's MI300X picture: four XCD pairs on four I/O dies in a 2x2 grid,
# tiers about 707 / 817 / 926 cycles for local / adjacent / opposite.
MI300X_GROUPS = (0, 0, 1, 1, 2, 2, 3, 3)
MI300X_DIST = ((0, 1, 1, 2), (1, 0, 2, 1), (1, 2, 0, 1), (2, 1, 1, 0))
MI300X_TIERS = (707, 817, 926)


def planted_latency(seed: int, n_samples: int, grp=MI300X_GROUPS, dist=MI300X_DIST,
                    tiers=MI300X_TIERS, common: int = 40, jitter: int = 12):
    """Returns (lat uint32 [n_xcds, n_samples], home int64 [n_samples])."""
    import numpy as np
    g = torch.Generator(device="cpu").manual_seed(seed)
    n_g = len(dist)
    home = torch.randint(0, n_g, (n_samples,), generator=g)
    off = torch.randint(0, max(1, common), (n_samples,), generator=g)
    jit = torch.randint(0, max(1, jitter), (len(grp), n_samples), generator=g)
    tier_t = torch.tensor([[tiers[dist[a][b]] for b in range(n_g)] for a in range(n_g)])
    lat = torch.stack([tier_t[grp[x]][home] for x in range(len(grp))]) + off + jit
    return lat.numpy().astype(np.uint32), home.numpy()


# Synthetic inputs for the partition-hash (interleave) discovery, host-only
# tests.  interleave_layout draws the probe's address blocks: a base line
# uniform among the 128-byte lines below 2^hi_bit, the base with each bit in
# [lo_bit, hi_bit) flipped, then n_pairs variants with two distinct such bits
# flipped.  planted_interleave_latency gives every address a home partition
# from a planted rule and the per-XCD latencies that go with it (two XCD halves,
# local / remote tiers as measured on MI355X, shared per-address offset and
# per-(XCD, address) jitter as in planted_latency).  Rules:
#   "xor": parity of (offset & mask & (2^page_bits - 1)), XOR a seeded bit per
#          2^page_bits page (the page's unknown physical bits);
#   "mixed": bit m0 XOR (bit m1 AND bit m2) of the three lowest mask bits, XOR
#          the page bit (not one parity: flips of m1, m2 change the home for
#          half of the addresses).
def interleave_layout(seed: int, n_bases: int, lo_bit: int, hi_bit: int, n_pairs: int):
    g = torch.Generator(device="cpu").manual_seed(seed)
    nb = hi_bit - lo_bit
    offs = []
    for _ in range(n_bases):
        base = int(torch.randint(0, 1 << (hi_bit - 7), (1,), generator=g)) << 7
        offs.append(base)
        offs.extend(base ^ (1 << b) for b in range(lo_bit, hi_bit))
        for _ in range(n_pairs):
            i, j = (int(v) + lo_bit for v in torch.randperm(nb, generator=g)[:2])
            offs.append(base ^ (1 << i) ^ (1 << j))
    return offs, 1 + nb + n_pairs


def planted_interleave_latency(seed: int, offs, mask: int, page_bits: int = 21, rule: str = "xor",
                               grp=(0, 0, 0, 0, 1, 1, 1, 1), tiers=(735, 950), common: int = 40,
                               jitter: int = 12):
    """Returns (lat uint32 [n_xcds, n_addr], home list)."""
    import numpy as np
    g = torch.Generator(device="cpu").manual_seed(seed)
    page_bit = {}
    home = []
    low = mask & ((1 << page_bits) - 1)
    mb = [b for b in range(64) if (mask >> b) & 1]
    for o in offs:
        p = o >> page_bits
        if p not in page_bit:
            page_bit[p] = int(torch.randint(0, 2, (1,), generator=g))
        if rule == "xor":
            h = bin(o & low).count("1") & 1
        elif rule == "mixed":
            h = ((o >> mb[0]) & 1) ^ (((o >> mb[1]) & 1) & ((o >> mb[2]) & 1))
        else:
            raise ValueError(rule)
        home.append(h ^ page_bit[p])
    n = len(offs)
    off = torch.randint(0, max(1, common), (n,), generator=g)
    jit = torch.randint(0, max(1, jitter), (len(grp), n), generator=g)
    h = torch.tensor(home)
    lat = torch.stack([torch.where(h == grp[x], tiers[0], tiers[1]) for x in range(len(grp))]) + off + jit
    return lat.numpy().astype(np.uint32), home


# Home-map inputs for host-only tests: a region of n_pages 2 MiB pages whose
# lines have a planted home, parity(offset & mask) XOR a seeded bit per page
# (the page's higher physical bits), and the per-XCD latencies of each page's
# first line and of n_verify random lines (two XCD halves, planted tiers as in
# planted_interleave_latency).  Returns (page-line latencies [n_xcds, n_pages],
# verify offsets, verify latencies [n_xcds, n_verify], planted home of a byte
# offset as a function).
def planted_home_region(seed: int, n_pages: int, mask: int, n_verify: int = 64,
                        grp=(0, 0, 0, 0, 1, 1, 1, 1), tiers=(735, 950), jitter: int = 12):
    import numpy as np
    g = torch.Generator(device="cpu").manual_seed(seed)
    page_bit = [int(v) for v in torch.randint(0, 2, (n_pages,), generator=g)]
    low = mask & ((2 << 20) - 1)

    def home_of(off: int) -> int:
        return (bin(off & low).count("1") & 1) ^ page_bit[off >> 21]

    def lat_of(offs):
        h = torch.tensor([home_of(o) for o in offs])
        jit = torch.randint(0, max(1, jitter), (len(grp), len(offs)), generator=g)
        return (torch.stack([torch.where(h == grp[x], tiers[0], tiers[1]) for x in range(len(grp))])
                + jit).numpy().astype(np.uint32)

    pages = [p << 21 for p in range(n_pages)]
    vo = [int(v) * 128 for v in torch.randint(0, n_pages << 14, (n_verify,), generator=g)]
    return lat_of(pages), vo, lat_of(vo), home_of


# Decode attention (Section 7.1 attention workloads; Appendix F): one query
# token per request, head dimension 128, 32 query heads against 32 key/value
# heads (multi-head) or 8 (grouped-query), batch 1..64, KV length from 512
# doubling.  Recipe: one torch CPU generator per problem seeded `seed`, q then
# K then V drawn N(0, 1) in fp32 in their storage shapes and rounded to bf16.
# Layout: q [B, H_q, D], K and V [B, H_kv, S_k, D] (each request's head a
# contiguous S_k x D slab).  The logical KV working set is 4 B S_k H_kv D bytes.
@dataclass(frozen=True)
class AttnProblem:
    name: str
    B: int
    Hq: int
    Hkv: int
    S: int
    D: int = 128
    seed: int = 6

    @property
    def kv_bytes(self) -> int:
        return 4 * self.B * self.S * self.Hkv * self.D

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)


def attn_problem(kind: str, B: int, S: int, seed: int = 6) -> AttnProblem:
    Hkv = {"mha": 32, "gqa": 8}[kind]
    return AttnProblem(f"decode_{kind}_B{B}_S{S}", B, 32, Hkv, S, seed=seed)


def make_attn_inputs(p: AttnProblem):
    """(q [B, H_q, D], K [B, H_kv, S, D], V [B, H_kv, S, D]) bf16 CPU tensors."""
    g = torch.Generator(device="cpu").manual_seed(p.seed)
    q = torch.randn((p.B, p.Hq, p.D), generator=g).to(torch.bfloat16)
    k = torch.randn((p.B, p.Hkv, p.S, p.D), generator=g).to(torch.bfloat16)
    v = torch.randn((p.B, p.Hkv, p.S, p.D), generator=g).to(torch.bfloat16)
    return q, k, v


def make_attn_inputs_on(p: AttnProblem, device):
    """Same shapes and distribution drawn on `device` (timing runs at full size)."""
    g = torch.Generator(device=device).manual_seed(p.seed)
    q = torch.randn((p.B, p.Hq, p.D), generator=g, device=device).to(torch.bfloat16)
    k = torch.randn((p.B, p.Hkv, p.S, p.D), generator=g, device=device).to(torch.bfloat16)
    v = torch.randn((p.B, p.Hkv, p.S, p.D), generator=g, device=device).to(torch.bfloat16)
    return q, k, v


def page_pool(x, table, pool_pages: int, fill: float = 0.0):
    """The pool a paged cache reads: x [B, H_kv, S, 128] (keys or values) laid
    out in 32-token pages at the pool pages `table` [B, H_kv, ceil(S / 32)]
    names (int32, any device); the tail of a head's last page and every pool
    page no entry names hold `fill`.  Returns bf16 [pool_pages, 32, 128] on
    x's device."""
    B, H, S, D = x.shape
    pph = (S + 31) // 32
    padded = torch.full((B, H, pph * 32, D), fill, dtype=x.dtype, device=x.device)
    padded[:, :, :S] = x
    pool = torch.full((pool_pages, 32, D), fill, dtype=x.dtype, device=x.device)
    idx = torch.as_tensor(table, device=x.device).reshape(-1).long()
    pool[idx] = padded.reshape(B * H * pph, 32, D)
    return pool


# Multi-head latent attention, decode (Section 7.1 attention workloads;
# Appendix F counts one compressed row of 512 + 64 values per token).  One
# query token per request; query heads 16 (a tensor-parallel shard of a
# 128-head model) or 128; each request caches one 576-wide row per token
# (512 latent values, which are also the value, then 64 rotary key values).
# Recipe: one torch CPU generator per problem seeded `seed`, q then the cache
# drawn N(0, 1) in fp32 in their storage shapes and rounded to bf16.  Layout:
# q [B, H_q, 576], cache [B, S_k, 576], O [B, H_q, 512].  The scale is
# 1 / sqrt(192), the per-head query-key width before the projections are
# absorbed (128 non-rotary + 64 rotary).  Working set 2 B S_k (512 + 64) bytes.
MLA_D_QK = 576
MLA_D_V = 512


@dataclass(frozen=True)
class MlaProblem:
    name: str
    B: int
    Hq: int
    S: int
    seed: int = 7

    @property
    def kv_bytes(self) -> int:
        return 2 * self.B * self.S * MLA_D_QK

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(192.0)


def mla_problem(B: int, Hq: int, S: int, seed: int = 7) -> MlaProblem:
    return MlaProblem(f"mla_decode_B{B}_H{Hq}_S{S}", B, Hq, S, seed=seed)


def make_mla_inputs(p: MlaProblem):
    """(q [B, H_q, 576], cache [B, S_k, 576]) bf16 CPU tensors."""
    g = torch.Generator(device="cpu").manual_seed(p.seed)
    q = torch.randn((p.B, p.Hq, MLA_D_QK), generator=g).to(torch.bfloat16)
    kv = torch.randn((p.B, p.S, MLA_D_QK), generator=g).to(torch.bfloat16)
    return q, kv


def make_mla_inputs_on(p: MlaProblem, device):
    """Same shapes and distribution drawn on `device` (timing runs at full size)."""
    g = torch.Generator(device=device).manual_seed(p.seed)
    q = torch.randn((p.B, p.Hq, MLA_D_QK), generator=g, device=device).to(torch.bfloat16)
    kv = torch.randn((p.B, p.S, MLA_D_QK), generator=g, device=device).to(torch.bfloat16)
    return q, kv
