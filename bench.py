#!/usr/bin/env python3
"""Benchmark of the hot path: persistent XCD-aware bf16 GEMM on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu] [--studies ...]

Workload: square bf16 GEMM M = N = K = 8192, inputs uniform[-1,1] from seed 1,
B stored [N][K], fp32 accumulation, bf16 output, on the whole GPU; the
topology probe runs first (untimed).  One step is one launch of the
persistent GEMM with the XCD-aware mapping (the schedule is cached after the
first launch).  W warm-up launches and a few seconds of untimed launches
(the clock and power state settle) precede the K timed steps.

Studies added to the same line (all on synthetic inputs): the three mappings
timed interleaved at 8192^3; the decoder-layer shapes; prefill || decode on
XCD-aligned and CU-striped partitions; the GEMM 4096^3 on 32 random and 2
XCD-aligned 128-CU sets beside a second tenant, with the max/min spread.

Prints one JSON line with the metric, the roofline of the GEMM kernel
(achieved TFLOP/s from HIP events around every launch, against the 2516.6
TFLOP/s dense bf16 peak), and the CPU oracle timed on a bounded sample of the
same problem on this host's cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from typing import Optional

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # 256 CU x 4096 flop/clk x 2.4 GHz, dense bf16 MFMA
HBM_PEAK_GBS = 8000.0
METRIC = "bf16 GEMM TFLOP/s (%MFMA peak): XCD-aware vs oblivious; CU-mask perf spread"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_bf16_persistent_square_8192_traffic.json")
GEMM_SRC = os.path.join(ROOT, "paper_2609_24270_amd", "csrc", "gemm.hip")


def kernel_source_hash() -> str:
    with open(GEMM_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source; otherwise None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("gemm_src_sha256_16") != kernel_source_hash():
        return None
    return t.get("bytes_per_launch")


def time_launches(fn, steps: int, stream):
    """Run fn() `steps` times on `stream`; return (total ms, mean per-launch ms)
    from HIP events recorded on that stream around the whole loop and around
    every launch."""
    import torch
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(2 * steps)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(steps):
        evs[2 * i].record(stream)
        fn()
        evs[2 * i + 1].record(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    total = e0.elapsed_time(e1)
    per = [evs[2 * i].elapsed_time(evs[2 * i + 1]) for i in range(steps)]
    return total, sum(per) / len(per)


def cpu_baseline(A, B, rows: int, C_gpu=None):
    """The oracle timed on the host's cores over rows 0..rows-1 of the
    problem.  When the GPU's output of the same problem is given, the oracle's
    rows (computed anyway) also check it: the gate is max |C - R32| /
    max(|R32|, rms(R32)) <= 2e-2 over every checked element, R32 being the
    oracle's fp32 sum before rounding."""
    import numpy as np
    import torch

    import oracle
    bits = lambda t: t.contiguous().view(torch.int16).numpy().view(np.uint16)
    Ab, Bb = bits(A[:rows]), bits(B)
    t0 = time.perf_counter()
    R, Co = oracle.gemm_bf16(Ab, Bb, "nk", want_r32=C_gpu is not None)
    dt = time.perf_counter() - t0
    flops = 2.0 * rows * B.shape[0] * B.shape[1]
    out = {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
           "kind": "oracle", "seconds": dt,
           "sample": f"rows 0..{rows - 1} of A against all of B (M={rows}, N={B.shape[0]}, K={B.shape[1]}), "
                     f"{flops / 1e9:.1f} GFLOP"}
    if C_gpu is None:
        return out, None
    Cg = bits(C_gpu[:rows])
    g = (Cg.astype(np.uint32) << 16).view(np.float32).astype(np.float64)  # bf16 bits -> value
    r = R.astype(np.float64)
    rms = float(np.sqrt(np.mean(r * r)))
    err = float(np.max(np.abs(g - r) / np.maximum(np.abs(r), rms)))
    parity = {"checked": f"rows 0..{rows - 1}, every column ({rows * B.shape[0]} elements)",
              "max_rel_err": err, "gate": 2e-2, "pass": err <= 2e-2,
              "bitwise_equal_to_oracle_frac": float(np.mean(Cg == Co))}
    return out, parity


def full_parity(A, B, C_gpu) -> dict:
    """Every output of one GPU product against the oracle (same gate as the
    CPU-baseline leg): max |C - R32| / max(|R32|, rms(R32)) over all elements,
    and the share bitwise equal to the oracle's rounded output."""
    import numpy as np
    import torch

    import oracle
    bits = lambda t: t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    t0 = time.perf_counter()
    R, Co = oracle.gemm_bf16(bits(A), bits(B), "nk", want_r32=True)
    dt = time.perf_counter() - t0
    Cg = bits(C_gpu)
    g = (Cg.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    r = R.astype(np.float64)
    rms = float(np.sqrt(np.mean(r * r)))
    err = float(np.max(np.abs(g - r) / np.maximum(np.abs(r), rms)))
    return {"elements": int(Cg.size), "max_rel_err": float(f"{err:.4e}"), "gate": 2e-2, "pass": err <= 2e-2,
            "bitwise_equal_to_oracle_frac": round(float(np.mean(Cg == Co)), 5), "oracle_s": round(dt, 2)}


def config_parity(topo, dev, stream) -> dict:
    """Full-output parity of every configuration's product, each launched the
    way the studies time it: 512^3, the three decoder shapes (full GPU, aware);
    prefill 8192x4096x4096 || decode 32x14336x4096 co-running on CU-striped
    sets; 4096^3 on the first seeded random 128-CU set beside the 64 MiB copy
    tenant (whose copy is checked too).  The 8192^3 headline is checked in the
    CPU-baseline leg."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    out = {}
    for p in (workloads.SQUARE_512,) + tuple(workloads.LLM_SHAPES):
        A, B = workloads.make_inputs(p)
        C = asym.gemm(A.to(dev), B.to(dev), topo=topo, stream=stream)
        torch.cuda.synchronize()
        out[p.name] = full_parity(A, B, C)
    (pa, pb), (da, db) = workloads.make_pd_inputs()
    pad, pbd, dad, dbd = pa.to(dev), pb.to(dev), da.to(dev), db.to(dev)
    cp = torch.empty((pa.shape[0], pb.shape[0]), dtype=torch.bfloat16, device=dev)
    cd = torch.empty((da.shape[0], db.shape[0]), dtype=torch.bfloat16, device=dev)
    prefill = topo.cuset(192, asym.CUSET_STRIPED)
    decode = [b for b in range(256) if b not in set(prefill)]
    asym.corun([asym.gemm_task(pad, pbd, cp, 1, "aware", mask=prefill),
                asym.gemm_task(dad, dbd, cd, 3, "aware", mask=decode)], topo)
    out["prefill_8192x4096x4096_striped_corun"] = full_parity(pa, pb, cp)
    out["decode_32x14336x4096_striped_corun"] = full_parity(da, db, cd)
    del pad, pbd, dad, dbd, cp, cd
    A, B = workloads.make_inputs(workloads.COLOC)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty((A.shape[0], B.shape[0]), dtype=torch.bfloat16, device=dev)
    src = workloads.copy_source(workloads.COPY_BYTES // 2).to(dev)
    dst = torch.zeros_like(src)
    m = workloads.random_mask_bits(workloads.COLOC.seed, 1, 128)[0]
    comp = [b for b in range(256) if b not in set(m)]
    asym.corun([asym.gemm_task(Ad, Bd, C, 3, "aware", mask=m), asym.copy_task(dst, src, 8, mask=comp)], topo)
    out["coloc_4096_random_set_copy_corun"] = full_parity(A, B, C)
    out["coloc_4096_random_set_copy_corun"]["copy_tenant_exact"] = bool(torch.equal(dst, src))
    out["all_pass"] = all(v["pass"] for v in out.values() if isinstance(v, dict)) and \
        out["coloc_4096_random_set_copy_corun"]["copy_tenant_exact"]
    return out


def clock_power(summ: dict, achieved_tflops: float) -> dict:
    """The sampler's figures and the MFMA fraction at the measured clock:
    achieved / (256 CUs x 4096 flop/clk x sclk)."""
    out = dict(summ)
    f = summ.get("sclk_mhz_mean")
    out["pct_peak_at_measured_clock"] = round(100.0 * achieved_tflops / (256 * 4096 * f * 1e6 / 1e12), 2) \
        if f else None
    return out


class ClockPowerSampler:
    """Shader clock and socket power read from the driver's hwmon files of the
    GPU's PCI function, sampled by a thread every `period` seconds while it
    runs (no GPU call).  Fields that cannot be read stay None."""

    def __init__(self, pci_bus_id: str, period: float = 0.02):
        import glob
        import threading
        self.period = period
        self.files = {}
        for d in sorted(glob.glob(f"/sys/bus/pci/devices/{pci_bus_id}/hwmon/hwmon*")):
            for name in ("power1_average", "power1_input", "freq1_input", "power1_cap"):
                f = os.path.join(d, name)
                if os.path.exists(f) and name not in self.files:
                    self.files[name] = f
        dpm = f"/sys/bus/pci/devices/{pci_bus_id}/pp_dpm_sclk"
        if "freq1_input" not in self.files and os.path.exists(dpm):
            self.files["pp_dpm_sclk"] = dpm
        self.samples = {k: [] for k in self.files}
        self._stop = threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True)

    def _read(self, name):
        try:
            with open(self.files[name]) as f:
                text = f.read()
            if name == "pp_dpm_sclk":
                # the current level is the line marked '*', e.g. "1: 1950Mhz *"; in Hz like freq1_input
                for ln in text.splitlines():
                    if ln.rstrip().endswith("*"):
                        return 1e6 * float(ln.split(":")[1].strip().lower().split("mhz")[0])
                return None
            return float(text.split()[0])
        except (OSError, ValueError, IndexError):
            return None

    def _run(self):
        while not self._stop.is_set():
            for k in self.files:
                if k == "power1_cap":
                    continue
                v = self._read(k)
                if v is not None:
                    self.samples[k].append(v)
            self._stop.wait(self.period)

    def __enter__(self):
        self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._t.join()

    def summary(self) -> dict:
        mean = lambda v: sum(v) / len(v) if v else None
        pw = self.samples.get("power1_average") or self.samples.get("power1_input") or []
        fr = self.samples.get("freq1_input") or self.samples.get("pp_dpm_sclk") or []
        cap = self._read("power1_cap") if "power1_cap" in self.files else None
        return {"sclk_mhz_mean": round(mean(fr) / 1e6, 1) if fr else None,
                "power_w_mean": round(mean(pw) / 1e6, 1) if pw else None,
                "power_cap_w": round(cap / 1e6, 1) if cap else None,
                "samples": len(fr) or len(pw),
                "source": ", ".join(sorted(self.files)) or "no hwmon file readable"}


def settle(fns, seconds: float):
    """Untimed launches, round-robin over fns, for `seconds` of wall time: the
    chip's clock and power state move for a second or more after a burst of
    GEMMs starts, and a measurement taken earlier would favour whichever
    variant runs last."""
    import torch
    t0 = time.perf_counter()
    n = 0
    while time.perf_counter() - t0 < seconds:
        for f in fns:
            f()
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def interleaved(fns: dict, rounds: int, stream) -> dict:
    """Mean per-launch ms of each fn, timed with HIP events on `stream`, the
    variants launched in turn within every round so that all of them see the
    same clock and power state."""
    import torch
    names = list(fns)
    evs = {k: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(rounds)] for k in names}
    torch.cuda.synchronize()
    for r in range(rounds):
        for k in names:
            evs[k][r][0].record(stream)
            fns[k]()
            evs[k][r][1].record(stream)
    torch.cuda.synchronize()
    return {k: sum(a.elapsed_time(b) for a, b in evs[k]) / rounds for k in names}


MAPPINGS = ("aware", "oblivious_grouped", "oblivious_rowmajor")


def affinity_halves(topo, n_xcds: int):
    """Two whole-XCD sets of equal size: the two measured affinity groups when the
    latency probe found exactly two of equal size, else the lower and upper XCDs."""
    g = topo.info()["group_of_xcd"]
    if g and min(g) >= 0 and sorted(set(g)) == [0, 1] and g.count(0) == g.count(1):
        a = sum(1 << x for x in range(n_xcds) if g[x] == 0)
    else:
        a = (1 << (n_xcds // 2)) - 1
    return a, ((1 << n_xcds) - 1) & ~a


def affinity_summary(topo):
    L = topo.latency()
    r = lambda v: [round(x, 1) for x in v]
    return {"n_samples": L["n_samples"], "passes": L["passes"], "clock_mhz": round(L["clock_mhz"], 1),
            "timer_overhead_cycles": L["timer_overhead"], "l2_hit_cycles": r(L["l2_hit"]),
            "mall_hit_cycles": r(L["mall_hit"]), "hbm_cycles": r(L["hbm"]),
            "group_of_xcd": L["group_of_xcd"], "home_share": [round(x, 4) for x in L["home_share"]],
            "unclassified_share": round(L["unclassified_share"], 4),
            "hbm_by_home_cycles": [r(v) for v in L["hbm_by_home"]]}


def llm_shapes(dev, stream, rounds: int):
    """Decoder-layer GEMMs M=4096 x (N,K) in {(14336,4096),(4096,14336),(6144,4096)},
    N(0,0.02) weights and N(0,1) activations, full GPU, the three mappings."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    out = {}
    for p in workloads.LLM_SHAPES:
        A, B = workloads.make_inputs(p)
        Ad, Bd = A.to(dev), B.to(dev)
        C = torch.empty((p.M, p.N), dtype=torch.bfloat16, device=dev)
        fns = {m: (lambda m=m: asym.gemm(Ad, Bd, C, mapping=m, stream=stream)) for m in MAPPINGS}
        settle(list(fns.values()), 0.3)
        ms = interleaved(fns, rounds, stream)
        out[p.name] = {"M": p.M, "N": p.N, "K": p.K,
                       **{m: round(p.flops / (ms[m] * 1e-3) / 1e12, 2) for m in MAPPINGS}}
    return out


def square_512(topo, dev, stream, launches: int = 50, rounds: int = 8):
    """512^3 (uniform[-1,1], seed 0) on the full GPU: the three mappings, each
    launch short enough that launches are queued behind a spin kernel and
    averaged; 128 x 128 tiles (16 tiles)."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    A, B = workloads.make_inputs(workloads.SQUARE_512)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty((512, 512), dtype=torch.bfloat16, device=dev)
    fns = {m: (lambda m=m: asym.gemm(Ad, Bd, C, mapping=m, topo=topo, stream=stream)) for m in MAPPINGS}
    for f in fns.values():
        f()
    ms = queued(fns, launches, rounds, stream)
    plan = asym.gemm_plan(Ad, Bd, C, topo=topo, stream=stream)
    return {"tile": [plan["tile_m"], plan["tile_n"]], "tiles": plan["tiles_m"] * plan["tiles_n"],
            **{m: {"us": round(1e3 * ms[m], 2), "tflops": round(2 * 512 ** 3 / (ms[m] * 1e-3) / 1e12, 2)}
               for m in MAPPINGS}}


DECODE_SHAPES = ((32, 4096, 4096), (64, 4096, 4096), (32, 6144, 4096), (32, 4096, 14336), (32, 14336, 4096),
                 (32, 10240, 4096), (128, 4096, 4096), (128, 14336, 4096))


def decode_projections(dev, stream, launches: int = 20, rounds: int = 5) -> list:
    """Decode-time projections (M = 32 to 128 rows of activations against a
    weight matrix) on the small-M kernel, with its plan (column-tile width,
    K ranges), and on the persistent kernel (aware); weights N(0, 0.02) and
    activations N(0, 1) drawn on the GPU from seed 3; the weight-streaming rate
    2 N K / time."""
    import torch

    import paper_2609_24270_amd as asym
    out = []
    for (M, N, K) in DECODE_SHAPES:
        g = torch.Generator(device=dev).manual_seed(3)
        A = torch.randn((M, K), generator=g, device=dev).to(torch.bfloat16)
        B = (torch.randn((N, K), generator=g, device=dev) * 0.02).to(torch.bfloat16)
        C = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        plan = asym.gemm_plan(A, B, C)
        f = lambda: asym.gemm(A, B, C, stream=stream)
        f()
        t = {"small_m": queued({"s": f}, launches, rounds, stream)["s"]}
        prev = asym.set_small_m(False)
        try:
            f()
            t["persistent"] = queued({"p": f}, launches, rounds, stream)["p"]
        finally:
            asym.set_small_m(prev)
        wbytes = 2 * N * K
        out.append({"M": M, "N": N, "K": K, "tile_n": plan["tile_n"], "tiles_n": plan["tiles_n"],
                    "k_splits": plan["k_splits"],
                    **{k: {"us": round(1e3 * v, 2), "weights_TBps": round(wbytes / (v * 1e-3) / 1e12, 3)}
                       for k, v in t.items()}})
        del A, B, C
    return out


def decode_gemm(dev, stream, launches: int = 20, rounds: int = 5):
    """Decode projection 32 x 14336 x 4096 (N(0,0.02) weights, N(0,1) activations)
    on the full GPU: the small-M kernel and the persistent kernel (aware), and
    the weight-streaming rate 2 N K / time."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    (_, _), (da, db) = workloads.make_pd_inputs()
    A, B = da.to(dev), db.to(dev)
    C = torch.empty((A.shape[0], B.shape[0]), dtype=torch.bfloat16, device=dev)
    small = lambda: asym.gemm(A, B, C, stream=stream)
    small()
    out = {"small_m": queued({"s": small}, launches, rounds, stream)["s"]}
    prev = asym.set_small_m(False)
    try:
        pers = lambda: asym.gemm(A, B, C, stream=stream)
        pers()
        out["persistent_aware"] = queued({"p": pers}, launches, rounds, stream)["p"]
    finally:
        asym.set_small_m(prev)
    wbytes = 2 * B.shape[0] * B.shape[1]
    return {k: {"us": round(1e3 * v, 2), "weights_TBps": round(wbytes / (v * 1e-3) / 1e12, 3),
                "tflops": round(2 * 32 * 14336 * 4096 / (v * 1e-3) / 1e12, 2)} for k, v in out.items()}


GRID_SHAPES = ((8192, 5120, 8192), (8192, 6656, 8192), (8192, 9216, 8192), (8192, 10240, 8192),
               (6144, 6144, 8192), (8192, 8192, 8192))


def grid_study(topo, dev, stream, launches: int = 20, settle_s: float = 1.0) -> list:
    """Tile-column counts that are not multiples of 8 (so round-robin dealing
    of a row-major order scatters each XCD's tiles): the three mappings,
    interleaved, `launches` each after `settle_s` of settling launches; inputs
    uniform[-1,1] from seed 1."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    out = []
    for (M, N, K) in GRID_SHAPES:
        p = workloads.make_problem(M, N, K, seed=1)
        A, B = workloads.make_inputs(p)
        Ad, Bd = A.to(dev), B.to(dev)
        C = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        fns = {m: (lambda m=m: asym.gemm(Ad, Bd, C, mapping=m, topo=topo, stream=stream)) for m in MAPPINGS}
        plan = asym.gemm_plan(Ad, Bd, C, mapping="aware", topo=topo, stream=stream)
        for f in fns.values():
            f()
        settle(list(fns.values()), settle_s)
        ms = interleaved(fns, launches, stream)
        out.append({"M": M, "N": N, "K": K, "tile_n": plan["tile_n"], "tiles": [plan["tiles_m"], plan["tiles_n"]],
                    **{m: round(p.flops / (ms[m] * 1e-3) / 1e12, 1) for m in ms}})
        del Ad, Bd, C
    return out


LARGE_SHAPES = ((16384, 16384, 16384), (16384, 15360, 16384), (16384, 15616, 16384), (12288, 12288, 12288))


def large_study(topo, dev, stream, launches: int = 6, settle_s: float = 1.0) -> list:
    """Products whose operands (384-512 MiB each) exceed the 256 MB memory-side
    cache, so that L2 misses are served from HBM: the three mappings,
    interleaved, `launches` each after `settle_s` of settling launches; inputs
    uniform[-1, 1] drawn on the GPU from seed 1 (A, then B)."""
    import torch

    import paper_2609_24270_amd as asym
    out = []
    for (M, N, K) in LARGE_SHAPES:
        g = torch.Generator(device=dev).manual_seed(1)
        Ad = (torch.rand((M, K), generator=g, device=dev) * 2 - 1).to(torch.bfloat16)
        Bd = (torch.rand((N, K), generator=g, device=dev) * 2 - 1).to(torch.bfloat16)
        C = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        fns = {m: (lambda m=m: asym.gemm(Ad, Bd, C, mapping=m, topo=topo, stream=stream)) for m in MAPPINGS}
        plan = asym.gemm_plan(Ad, Bd, C, mapping="aware", topo=topo, stream=stream)
        for f in fns.values():
            f()
        settle(list(fns.values()), settle_s)
        ms = interleaved(fns, launches, stream)
        flops = 2.0 * M * N * K
        out.append({"M": M, "N": N, "K": K, "tile_n": plan["tile_n"], "tiles": [plan["tiles_m"], plan["tiles_n"]],
                    **{m: round(flops / (ms[m] * 1e-3) / 1e12, 1) for m in ms},
                    "aware_vs_grouped": round(ms["oblivious_grouped"] / ms["aware"], 4),
                    "aware_vs_rowmajor": round(ms["oblivious_rowmajor"] / ms["aware"], 4)})
        del Ad, Bd, C
        torch.cuda.empty_cache()
    return out


def pd_sets(topo, halves):
    """The prefill / decode CU sets: 192 striped bits and the other 64; the
    XCD-aligned split with the decode pair taken from one affinity group."""
    import paper_2609_24270_amd as asym
    prefill = topo.cuset(192, asym.CUSET_STRIPED)
    decode = [b for b in range(256) if b not in set(prefill)]
    grp = [x for x in range(8) if (halves[1] >> x) & 1]
    dec_x = (1 << grp[-1]) | (1 << grp[-2])
    pre_x = 0xFF & ~dec_x
    pre_m, dec_m = topo.cuset_split_xcds(pre_x)
    return prefill, decode, pre_x, dec_x, pre_m, dec_m


def trace_summary(t: dict, khz: int, t0: Optional[int] = None) -> dict:
    """Per-XCD summary of one traced GEMM launch; times in microseconds from
    t0 (default: the first workgroup's start).  A CU is told apart by bits
    8-15 of HW_ID (CU, shader array and engine numbers)."""
    import numpy as np
    t0 = int(t["start"].min()) if t0 is None else t0
    rel = lambda v: (v.astype(np.int64) - t0) * (1e3 / khz)
    st, ft, en = rel(t["start"]), rel(t["first_tile"]), rel(t["end"])
    w = t["worked"] == 1
    live = np.maximum(1, (t["end"] - t["start"]).astype(np.int64))
    mhz = t["cycles"].astype(np.float64) * khz / live / 1e3  # shader clock over each workgroup's life
    cu = (t["hw_id"] >> 8) & 0xFF
    per = []
    for x in range(8):
        s = t["xcc"] == x
        sw, ex = s & w, s & ~w
        d = {"workgroups": int(s.sum()), "workers": int(sw.sum()), "tiles": int(t["tiles"][s].sum()),
             "cus_used": int(len(np.unique(cu[s])))}
        if sw.any():
            d.update(last_start_us=round(float(st[sw].max()), 1), first_tile_by_us=round(float(ft[sw].max()), 1),
                     first_end_us=round(float(en[sw].min()), 1), last_end_us=round(float(en[sw].max()), 1),
                     us_per_tile=round(float(((en[sw] - ft[sw]) / t["tiles"][sw]).mean()), 2),
                     clock_mhz=round(float(mhz[sw].mean()), 0))
            d["kcycles_per_tile"] = round(d["us_per_tile"] * d["clock_mhz"] / 1e3, 1)
        if ex.any():
            d["exit_only_starts_us"] = [round(float(v), 1) for v in np.sort(st[ex])][:8]
            d["exit_only_last_end_us"] = round(float(en[ex].max()), 1)
        per.append(d)
    worked = t["tiles"][w]
    return {"grid": int(len(t["tiles"])), "first_start_us": round(float(st.min()), 1),
            "span_us": round(float(en.max() - st.min()), 1), "last_end_us": round(float(en.max()), 1),
            "tiles_per_worker": {int(k): int(v) for k, v in zip(*np.unique(worked, return_counts=True))},
            "mean_us_per_tile": round(float(((en[w] - ft[w]) / worked).mean()), 2),
            "mean_clock_mhz": round(float(mhz[w].mean()), 0),
            "per_xcd": per}


def array_balance(t: dict, topo, mask, khz: int) -> list:
    """Per XCD and shader array (engine * 2 + array, from HW_ID): the mask's
    CUs there, the workgroups that started within 5 us of the launch's first
    start, and those that started later (they waited for a CU)."""
    import numpy as np
    cus = topo.json()["cus"]  # [xcc, se, sh, cu, mask bit]
    bits = set(range(256)) if mask is None else set(mask)
    arr = lambda se, sh: se * 2 + sh
    n_arr = 1 + max(arr(c[1], c[2]) for c in cus)
    rel = (t["start"].astype(np.int64) - int(t["start"].min())) * (1e3 / khz)
    se, sh = (t["hw_id"] >> 13) & 0x7, (t["hw_id"] >> 12) & 0x1
    out = []
    for x in range(8):
        m = [0] * n_arr
        for c in cus:
            if c[0] == x and c[4] in bits:
                m[arr(c[1], c[2])] += 1
        sel = t["xcc"] == x
        early = [int(np.sum(sel & (rel < 5.0) & (arr(se, sh) == a))) for a in range(n_arr)]
        late = [int(np.sum(sel & (rel >= 5.0) & (arr(se, sh) == a))) for a in range(n_arr)]
        out.append({"mask_cus": m, "started_at_launch": early, "started_late": late})
    return out


def pd_trace(topo, dev, halves, launches: int = 10, traced: int = 4, warm_ms=(0, 20, 500)):
    """The prefill GEMM 8192x4096x4096 alone, aware, on the XCD-aligned set
    (6 XCDs, claiming form) and on the 192 striped CUs (static form), plus the
    full chip: untraced ms per launch from the co-run executor (launched from
    native code, as the co-run studies time it), then for each warm-up length
    (ms of untraced launches queued just before, after 50 ms idle) `traced`
    traced launches queued back to back.  Each warm-up gets the last traced
    launch's span and mean shader clock; the longest one also its per-XCD
    summary, the shader-array balance and the gaps between one launch's last
    workgroup end and the next launch's first start."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    (pa, pb), _ = workloads.make_pd_inputs()
    pa, pb = pa.to(dev), pb.to(dev)
    cp = torch.empty((pa.shape[0], pb.shape[0]), dtype=torch.bfloat16, device=dev)
    prefill, _, pre_x, _, pre_m, _ = pd_sets(topo, halves)
    khz = asym.device_query(0)["wall_clock_khz"]
    tick = 1e3 / khz
    sets = {"xcd_aligned": (pre_m, pre_x), "cu_striped": (prefill, 0), "full_chip": (None, 0)}
    out = {}
    for name, (mask, xm) in sets.items():
        asym.corun([asym.gemm_task(pa, pb, cp, 3, "aware", mask=mask, xcd_mask=xm)], topo)
        ms = asym.corun([asym.gemm_task(pa, pb, cp, launches, "aware", mask=mask, xcd_mask=xm)], topo)[0]["ms_per_iter"]
        s = asym.stream_create(topo, mask) if mask is not None else torch.cuda.current_stream()
        try:
            asym.gemm_trace(pa, pb, cp, topo=topo, xcd_mask=xm, stream=s)  # load the traced kernel
            warm = {}
            for w in warm_ms:
                time.sleep(0.05)
                for _ in range(int(w / ms) if w else 0):
                    asym.gemm(pa, pb, cp, topo=topo, xcd_mask=xm, stream=s)
                ts = asym.gemm_trace(pa, pb, cp, topo=topo, xcd_mask=xm, stream=s, launches=traced)
                r = trace_summary(ts[-1], khz)
                warm[w] = {"spans_us": [round((int(t["end"].max()) - int(t["start"].min())) * tick, 1) for t in ts],
                           "clock_mhz": r["mean_clock_mhz"]}
            r["gaps_us"] = [round((int(b["start"].min()) - int(a["end"].max())) * tick, 1) for a, b in zip(ts, ts[1:])]
            r["after_warm_up_ms"] = warm
            r["ms_per_launch"] = round(ms, 4)
            r["claims"] = ts[-1]["plan"]["claims"]
            r["mask_cus_per_xcd"] = topo.cuset_counts(mask) if mask is not None else None
            r["arrays"] = array_balance(ts[-1], topo, mask, khz)
            out[name] = r
        finally:
            if mask is not None:
                asym.stream_destroy(s)
    return out


def prefill_decode(topo, dev, iters: int, halves, warm: int = 0):
    """Prefill GEMM 8192x4096x4096 on 192 CUs co-running with decode GEMM
    32x14336x4096 on the other 64, on XCD-aligned sets (6 XCDs / 2 XCDs, the
    decode pair taken from one affinity group) and on CU-striped sets (24 / 8
    CUs of every XCD); aware mapping; each also alone on its set.  Every run
    first runs `warm` times its timed launches untimed (warm = 100: about
    300 ms), so the shader clock has risen under that run's own load."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    (pa, pb), (da, db) = workloads.make_pd_inputs()
    pa, pb, da, db = pa.to(dev), pb.to(dev), da.to(dev), db.to(dev)
    cp = torch.empty((pa.shape[0], pb.shape[0]), dtype=torch.bfloat16, device=dev)
    cd = torch.empty((da.shape[0], db.shape[0]), dtype=torch.bfloat16, device=dev)
    prefill, decode, pre_x, dec_x, pre_m, dec_m = pd_sets(topo, halves)
    pre = lambda mask, xm: asym.gemm_task(pa, pb, cp, iters, "aware", mask=mask, xcd_mask=xm, warm_iters=warm * iters)
    dec = lambda mask, xm: asym.gemm_task(da, db, cd, 3 * iters, "aware", mask=mask, xcd_mask=xm,
                                          warm_iters=warm * 3 * iters)
    sets = {"xcd_aligned": ((pre_m, pre_x), (dec_m, dec_x)), "cu_striped": ((prefill, 0), (decode, 0))}
    out = {}
    for _ in range(2):  # first round settles the clock; the second is kept
        for k, (ps, ds) in sets.items():
            r = asym.corun([pre(*ps), dec(*ds)], topo)
            p_alone, d_alone = asym.corun([pre(*ps)], topo)[0], asym.corun([dec(*ds)], topo)[0]
            out[k] = {"prefill_ms": round(r[0]["ms_per_iter"], 4), "prefill_tflops": round(r[0]["tflops"], 2),
                      "decode_ms": round(r[1]["ms_per_iter"], 4), "decode_tflops": round(r[1]["tflops"], 2),
                      "prefill_alone_ms": round(p_alone["ms_per_iter"], 4),
                      "decode_alone_ms": round(d_alone["ms_per_iter"], 4)}
    return out


READ_TENANT_PASSES = 100   # about 27 ms at 4 TB/s: longer than 20 GEMM launches beside it


def spread_study(topo, dev, n_masks: int, iters: int, halves, tenant: str = "copy", repeats: int = 5):
    """GEMM 4096^3 (uniform[-1,1], seed 4) on 128-CU sets: n_masks seeded random
    choices of 128 mask bits (what a topology-oblivious allocator hands out) and
    the two whole-XCD halves (the measured affinity groups; each side lends the
    other one CU per XCD and works only on its own XCDs).  A second tenant runs
    on the complementary 128 CUs: the 64 MiB bf16 streaming copy (tenant
    "copy", Section 7.3's co-located tenant; its pass count is set from solo
    runs so that it outlasts the GEMM), the same GEMM with three times the
    launches ("gemm"), or the whole-buffer reader making READ_TENANT_PASSES
    passes of 1 GiB ("read"), kept to its own XCDs on the aligned halves.
    Each (set, mapping) is co-run `repeats` times in a row and its median
    TFLOP/s kept; reported per mapping: the median, min and max of the per-set
    medians and their max/min spread, the largest max/min within one set's
    repeats, in how many runs the tenant ended after the GEMM (so that it ran
    beside every launch), and the GEMM alone on the first random set and on
    the halves (median of the repeats)."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    A, B = workloads.make_inputs(workloads.COLOC)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty((A.shape[0], B.shape[0]), dtype=torch.bfloat16, device=dev)
    C2 = torch.empty_like(C)
    rbuf = torch.ones(256 << 20, dtype=torch.float32, device=dev) if tenant == "read" else None
    src = workloads.copy_source(workloads.COPY_BYTES // 2).to(dev) if tenant == "copy" else None
    dst = torch.empty_like(src) if tenant == "copy" else None
    masks = workloads.random_mask_bits(workloads.COLOC.seed, n_masks, 128)
    med = lambda v: sorted(v)[len(v) // 2]
    copy_passes = 0
    if tenant == "copy":
        # passes: 2x the solo GEMM's time over the slowest solo copy pass on a complement
        m0 = masks[0]
        g_ms = max(asym.corun([asym.gemm_task(Ad, Bd, C, iters, mp, mask=m0)], topo)[0]["ms_total"]
                   for mp in MAPPINGS)
        c_ms = 0.0
        for m in masks[:4]:
            comp = [b for b in range(256) if b not in set(m)]
            c_ms = max(c_ms, asym.corun([asym.copy_task(dst, src, 10, mask=comp)], topo)[0]["ms_per_iter"])
        copy_passes = max(10, int(2.0 * g_ms / max(c_ms, 1e-3)) + 1)

    def other(cus, xm=0):
        if tenant == "read":
            return asym.read_task(rbuf, READ_TENANT_PASSES, mask=cus, xcd_mask=xm)
        if tenant == "copy":
            return asym.copy_task(dst, src, copy_passes, mask=cus, xcd_mask=xm)
        return asym.gemm_task(Ad, Bd, C2, 3 * iters, "aware", mask=cus, xcd_mask=xm)
    per = {m: [] for m in MAPPINGS}
    within = {m: 1.0 for m in MAPPINGS}
    tenant_rate = []
    counts = []
    runs, covered = 0, 0

    def cover(r):
        # the tenant was busy for the whole measurement when it ended last
        nonlocal runs, covered
        runs += 1
        covered += r[1]["ms_total"] >= r[0]["ms_total"]
    # settle: one untimed co-run on the first set
    comp0 = [b for b in range(256) if b not in set(masks[0])]
    asym.corun([asym.gemm_task(Ad, Bd, C, iters, "aware", mask=masks[0]), other(comp0)], topo)
    for i, m in enumerate(masks):
        comp = [b for b in range(256) if b not in set(m)]
        counts.append(topo.cuset_counts(m))
        for mapping in MAPPINGS:
            v = []
            for _ in range(repeats):
                r = asym.corun([asym.gemm_task(Ad, Bd, C, iters, mapping, mask=m), other(comp)], topo)
                v.append(r[0]["tflops"])
                if tenant != "gemm":
                    tenant_rate.append(r[1]["gbps"])
                cover(r)
            per[mapping].append(med(v))
            within[mapping] = max(within[mapping], max(v) / min(v))
    m0 = masks[0]
    alone = {mp: round(med([asym.corun([asym.gemm_task(Ad, Bd, C, iters, mp, mask=m0)], topo)[0]["tflops"]
                            for _ in range(repeats)]), 2) for mp in MAPPINGS}
    aligned, aligned_rate, aligned_alone, aligned_within = [], [], [], []
    for xm in halves:
        ma, mb = topo.cuset_split_xcds(xm)
        aligned_alone.append(round(med([asym.corun([asym.gemm_task(Ad, Bd, C, iters, "aware", mask=ma,
                                                                   xcd_mask=xm)], topo)[0]["tflops"]
                                        for _ in range(repeats)]), 2))
        v, rate = [], []
        for _ in range(repeats):
            r = asym.corun([asym.gemm_task(Ad, Bd, C, iters, "aware", mask=ma, xcd_mask=xm),
                            other(mb, 0xFF & ~xm)], topo)
            v.append(r[0]["tflops"])
            rate.append(r[1]["gbps"])
            cover(r)
        aligned.append(round(med(v), 2))
        aligned_within.append(round(max(v) / min(v), 4))
        aligned_rate.append(round(med(rate), 1))
    summ = {"tenant": tenant, "n_random_sets": n_masks, "iters": iters, "repeats_per_set": repeats,
            **({"copy_passes": copy_passes, "copy_bytes": workloads.COPY_BYTES} if tenant == "copy" else {}),
            "aligned_aware_tflops": aligned, "aligned_within_set_max_min": aligned_within,
            **({"aligned_tenant_GBps": aligned_rate,
                "random_tenant_GBps_median": round(med(tenant_rate), 1)} if tenant != "gemm" else {}),
            "tenant_outlasted_gemm": f"{covered}/{runs}",
            "alone_tflops": {"first_random_set": alone, "aligned_halves_aware": aligned_alone},
            "random_set_min_max_cus_per_xcd": [min(min(c) for c in counts), max(max(c) for c in counts)]}
    for mapping, v in per.items():
        summ[f"random_{mapping}"] = {"median": round(med(v), 2), "min": round(min(v), 2), "max": round(max(v), 2),
                                     "spread": round(max(v) / min(v), 4),
                                     "within_set_max_min": round(within[mapping], 4)}
    return summ


def balanced_study(topo, dev, iters: int = 20, repeats: int = 5, warm: int = 10):
    """Locality without balance: GEMM 4096^3 (uniform[-1,1], seed 4) on the
    striped 128-CU and 192-CU sets (16 and 24 CUs of every XCD, so every
    mapping gives each XCD the same work), alone and beside the 64 MiB
    streaming copy on the complementary CUs; each mapping `repeats` times,
    median kept, every co-run after `warm` times its launches (and a matching
    share of copy passes) of untimed warm-up.  Any gap between the mappings is
    what L2 locality is worth under the tenant's memory traffic."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    A, B = workloads.make_inputs(workloads.COLOC)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty((A.shape[0], B.shape[0]), dtype=torch.bfloat16, device=dev)
    src = workloads.copy_source(workloads.COPY_BYTES // 2).to(dev)
    dst = torch.empty_like(src)
    med = lambda v: sorted(v)[len(v) // 2]
    out = {}
    for n in (128, 192):
        cus = topo.cuset(n, asym.CUSET_STRIPED)
        comp = [b for b in range(256) if b not in set(cus)]
        g_ms = max(asym.corun([asym.gemm_task(Ad, Bd, C, iters, mp, mask=cus)], topo)[0]["ms_total"]
                   for mp in MAPPINGS)
        c_ms = asym.corun([asym.copy_task(dst, src, 10, mask=comp)], topo)[0]["ms_per_iter"]
        passes = max(10, int(2.0 * g_ms / max(c_ms, 1e-3)) + 1)
        row = {"cus_per_xcd": topo.cuset_counts(cus), "copy_passes": passes}
        for mp in MAPPINGS:
            alone = [asym.corun([asym.gemm_task(Ad, Bd, C, iters, mp, mask=cus, warm_iters=warm * iters)],
                                topo)[0]["tflops"] for _ in range(repeats)]
            co, rate, covered = [], [], 0
            for _ in range(repeats):
                r = asym.corun([asym.gemm_task(Ad, Bd, C, iters, mp, mask=cus, warm_iters=warm * iters),
                                asym.copy_task(dst, src, passes, mask=comp, warm_passes=warm * passes // 2)], topo)
                co.append(r[0]["tflops"])
                rate.append(r[1]["gbps"])
                covered += r[1]["ms_total"] >= r[0]["ms_total"]
            row[mp] = {"alone_tflops": round(med(alone), 2), "beside_copy_tflops": round(med(co), 2),
                       "copy_GBps": round(med(rate), 1), "copy_outlasted_gemm": f"{covered}/{repeats}",
                       "within_max_min": round(max(co) / min(co), 4)}
        for mp in ("oblivious_grouped", "oblivious_rowmajor"):
            row[f"aware_vs_{mp}"] = {k: round(row["aware"][k] / row[mp][k], 4)
                                     for k in ("alone_tflops", "beside_copy_tflops")}
        out[f"striped_{n}"] = row
    return out


def queued(fns: dict, launches: int, rounds: int, stream, warm_ms: float = 40.0) -> dict:
    """Mean per-launch ms of each fn for kernels too short to time from the
    host: each round parks the stream on a spin kernel while the host queues,
    behind it, untimed launches of every variant in turn adding up to about
    `warm_ms` of GPU work (at most 512 launches), then `launches` back-to-back
    launches of each variant, each batch bracketed by HIP events on the
    stream.  The chip's clock and power control settle only some 25-50 ms
    after an idle spell such as the one-wave spin: launches 2-8 ms after it
    ran up to 1.3x slower than 50 ms after it.  The spin lasts long enough for
    the host to queue every launch of the round behind it, so that none waits
    on the host.  The order of the batches rotates from round to round and the
    rounds are a multiple of the variant count, so every variant takes every
    position equally often."""
    import math
    import time

    import torch
    names = list(fns)
    n = len(names)
    rounds = -(-rounds // n) * n
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        a.record(stream)
        torch.cuda._sleep(1 << 20)
        b.record(stream)
    torch.cuda.synchronize()
    cycles_per_ms = (1 << 20) / max(a.elapsed_time(b), 1e-3)
    # GPU time of one launch of every variant, and the host's cost of a launch
    probe = 3
    a.record(stream)
    h0 = time.perf_counter()
    for _ in range(probe):
        for k in names:
            fns[k]()
    host_ms = (time.perf_counter() - h0) * 1e3 / (probe * n)
    b.record(stream)
    torch.cuda.synchronize()
    cycle_ms = max(a.elapsed_time(b) / probe, 1e-3)
    warm = max(launches, min(math.ceil(warm_ms / cycle_ms), max(launches, 512 // n)))
    spin = int(cycles_per_ms * max(8.0, 1.5 * host_ms * n * (warm + launches) + 2.0))
    evs = {k: [] for k in names}
    for r in range(rounds):
        order = names[r % n:] + names[:r % n]
        with torch.cuda.stream(stream):
            torch.cuda._sleep(spin)
        for _ in range(warm):
            for k in order:
                fns[k]()
        for k in order:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(launches):
                fns[k]()
            e1.record(stream)
            evs[k].append((e0, e1))
        torch.cuda.synchronize()
    return {k: sum(x.elapsed_time(y) for x, y in evs[k]) / (rounds * launches) for k in names}


def grouped_study(dev, stream, seeds, launches: int, rounds: int):
    """Grouped GEMM over the 16 expert-layer configurations, (G, M) x (N, K),
    five row-count seeds each (M_i = floor(M U_i), U_i ~ U(0.7, 1.3)): per
    instance, the three mappings timed in turn; reported per configuration
    (seed means) with the logical working set W = 2 (sum M_i (K + N) + G N K)
    bytes, and the aware speedups over all instances."""
    import math

    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    per, sp_g, sp_r = {}, [], []
    for base in workloads.GROUPED:
        rows = []
        for seed in seeds:
            p = workloads.grouped_problem(base.G, base.M, base.N, base.K, seed=seed)
            Ms, A, B = workloads.make_grouped_inputs_on(p, dev)
            C = torch.empty((sum(Ms), p.N), dtype=torch.bfloat16, device=dev)
            # the mappings are compared on the persistent kernel; groups of at
            # most 64 rows are also timed on the small-M kernel
            prev = asym.set_small_m(False)
            try:
                fns = {m: (lambda m=m: asym.gemm_grouped(A, B, Ms, C, mapping=m, stream=stream)) for m in MAPPINGS}
                for f in fns.values():
                    f()
                ms = queued(fns, launches, rounds, stream)
            finally:
                asym.set_small_m(prev)
            if max(Ms) <= 64:
                f = lambda: asym.gemm_grouped(A, B, Ms, C, stream=stream)
                f()
                ms["small_m"] = queued({"s": f}, launches, rounds, stream)["s"]
            rows.append((p.flops, p.working_set_bytes, ms))
            sp_g.append(ms["oblivious_grouped"] / ms["aware"])
            sp_r.append(ms["oblivious_rowmajor"] / ms["aware"])
            del A, B, C
        n = len(rows)
        gm = lambda v: math.exp(sum(math.log(x) for x in v) / len(v))
        per[f"G{base.G}_M{base.M}_N{base.N}_K{base.K}"] = {
            "W_GB": round(sum(r[1] for r in rows) / n / 1e9, 4),
            **{f"{m}_us": round(1e3 * sum(r[2][m] for r in rows) / n, 2) for m in MAPPINGS},
            "aware_tflops": round(sum(r[0] / (r[2]["aware"] * 1e-3) for r in rows) / n / 1e12, 1),
            "aware_TBps_W": round(sum(r[1] / (r[2]["aware"] * 1e-3) for r in rows) / n / 1e12, 3),
            "speedup_vs_oblivious_grouped": round(gm([r[2]["oblivious_grouped"] / r[2]["aware"] for r in rows]), 4),
            "speedup_vs_oblivious_rowmajor": round(gm([r[2]["oblivious_rowmajor"] / r[2]["aware"] for r in rows]), 4)}
        if "small_m" in rows[0][2]:
            e = per[f"G{base.G}_M{base.M}_N{base.N}_K{base.K}"]
            e["small_m_us"] = round(1e3 * sum(r[2]["small_m"] for r in rows) / n, 2)
            e["small_m_TBps_W"] = round(sum(r[1] / (r[2]["small_m"] * 1e-3) for r in rows) / n / 1e12, 3)
            e["small_m_speedup_vs_aware"] = round(gm([r[2]["aware"] / r[2]["small_m"] for r in rows]), 4)
    torch.cuda.empty_cache()

    def summ(v):
        v = sorted(v)
        return {"min": round(v[0], 4), "median": round(v[len(v) // 2], 4), "max": round(v[-1], 4),
                "geomean": round(math.exp(sum(math.log(x) for x in v) / len(v)), 4)}
    return {"seeds": list(seeds), "launches_per_run": launches, "rounds": rounds, "instances": len(sp_g),
            "aware_speedup_vs_oblivious_grouped": summ(sp_g),
            "aware_speedup_vs_oblivious_rowmajor": summ(sp_r), "per_config": per}


def interleave_summary(dev):
    """Partition-hash discovery over offset bits 7..33 of a 16 GiB allocation."""
    import paper_2609_24270_amd as asym
    r, *_ = asym.interleave_probe(0, n_bases=128, lo_bit=7, hi_bit=34, n_pairs=4, passes=4)
    bits = "".join({1: "1", 0: "0", -1: "?", -2: "."}[r["verdict"][b]] for b in range(7, 34))
    return {"hash_mask": hex(r["hash_mask"]), "lowest_bit": r["lowest_bit"], "granularity": r["granularity"],
            "determined_below": r["determined_below"], "verdicts_bits_7_to_33": bits,
            "pair_checks": r["pair_checks"], "pair_agree": r["pair_agree"],
            "unclassified_share": round(r["unclassified_share"], 4),
            "local_cycles": round(r["local_cycles"], 1), "remote_cycles": round(r["remote_cycles"], 1),
            "group_of_xcd": r["group_of_xcd"]}, r


def numa_bw_study(dev, hash_res, rounds: int = 3, gib: int = 16):
    """Read bandwidth of a 16 GiB region by chunk home: every chunk read once per
    iteration, each XCD reading chunks homed on its own group (local), on the
    other group (remote), or chunks in address order whatever their home (all);
    on the whole chip and on one group's XCDs alone."""
    import torch

    import paper_2609_24270_amd as asym
    nbytes = gib << 30
    page = 2 << 20
    raw = torch.empty(nbytes + page, dtype=torch.uint8, device=dev)
    shift = (-raw.data_ptr()) % page
    ptr = raw.data_ptr() + shift
    raw.fill_(1)
    chunk_log2 = max(12, hash_res["lowest_bit"])
    info, homes = asym.home_map(ptr, nbytes, hash_res["hash_mask"], chunk_log2,
                                group_of_xcd=hash_res["group_of_xcd"], passes=2, n_verify=4096, seed=7)
    grp = info["group_of_xcd"]
    g0 = sum(1 << x for x, g in enumerate(grp) if g == 0)
    cases = {}
    for where, xm in (("chip", 0), ("group0_xcds", g0)):
        for name, mode in (("all", asym.CHUNKS_ALL), ("local", asym.CHUNKS_LOCAL), ("remote", asym.CHUNKS_REMOTE)):
            cases[f"{where}_{name}"] = asym.chunk_lists(homes, len(grp), grp, mode, xm)
    acc = {k: 0.0 for k in cases}
    for _ in range(rounds):
        for k, (chunks, off) in cases.items():
            ms, _ = asym.chunk_read_bw(ptr, nbytes, chunk_log2, chunks, off, iters=5)
            acc[k] += len(chunks) * (1 << chunk_log2) / (ms * 1e-3) / 1e9
    # latency as the bound: few workgroups per XCD, each reading one chunk at a
    # time, over the first 2 GiB of the region (whole chip; local, remote and
    # address-order lists of the same chunks)
    import numpy as np
    limit = (2 << 30) >> chunk_log2
    low = {}
    for name, mode in (("all", asym.CHUNKS_ALL), ("local", asym.CHUNKS_LOCAL), ("remote", asym.CHUNKS_REMOTE)):
        chunks, off = asym.chunk_lists(homes, len(grp), grp, mode, 0)
        segs = [np.asarray(chunks[off[x]:off[x + 1]]) for x in range(len(grp))]
        segs = [g_[g_ < limit] for g_ in segs]
        low[name] = (np.concatenate(segs).astype(np.uint32), np.cumsum([0] + [len(g_) for g_ in segs]))
    lat = {}
    for w in (1, 4, 16, 64, 256):
        r = {}
        for name, (chunks, off) in low.items():
            ms, _ = asym.chunk_read_bw(ptr, nbytes, chunk_log2, chunks, off, iters=3, workers_per_xcd=w)
            r[name] = round(len(chunks) * (1 << chunk_log2) / (ms * 1e-3) / 1e9, 1)
        r["local_over_remote"] = round(r["local"] / r["remote"], 3)
        r["local_over_all"] = round(r["local"] / r["all"], 3)
        lat[f"workers_per_xcd_{w}"] = r
    del raw
    torch.cuda.empty_cache()
    return {"region_gib": gib, "chunk_bytes": 1 << chunk_log2, "rounds": rounds,
            "map": {k: info[k] for k in ("n_pages", "unclassified_pages", "chunk_share", "verify_classified",
                                         "verify_agree", "local_cycles", "remote_cycles")},
            "GBps": {k: round(v / rounds, 1) for k, v in acc.items()},
            "low_parallelism_GBps_first_2GiB": lat}


def placed_attention_study(dev, hres, topo, stream, launches: int = 20, rounds: int = 5):
    """Decode attention (GQA 32 / 8 heads, head dim 128) over a paged cache
    whose pages are placed by home (Appendix E): each task's pages homed on
    the die of the XCD that owns the task (local), on the other die (remote),
    or in address order (in order: pages alternate homes as the partition hash
    deals them); the dense call beside them.  B = 1 and 4, S = 8192 and 32768,
    on the whole chip and on one die's four XCDs (whole-XCD restriction).
    Pages of 8 KiB are the chunks the home map measures."""
    import numpy as np
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    grp = list(hres["group_of_xcd"])
    g0 = sum(1 << x for x, g in enumerate(grp) if g == 0)
    page = asym.PAGE_TOKENS * 128 * 2
    out = {}
    for B, S in ((1, 8192), (1, 32768), (4, 8192)):
        p = workloads.AttnProblem(f"placed_B{B}_S{S}", B, 32, 8, S, seed=12)
        q, k, v = workloads.make_attn_inputs_on(p, dev)
        pph = -(-S // asym.PAGE_TOKENS)
        n = B * 8 * pph
        P = -(-(2 * n + 2048) // 256) * 256         # pool pages per pool, a whole number of 2 MiB pages
        raw = torch.empty(2 * P * page + (2 << 20), dtype=torch.uint8, device=dev)
        shift = (-raw.data_ptr()) % (2 << 20)
        base = raw.data_ptr() + shift
        info, homes = asym.home_map(base, 2 * P * page, hres["hash_mask"], 13, group_of_xcd=grp, passes=2,
                                    n_verify=512, seed=7)
        pools = raw[shift: shift + 2 * P * page].view(torch.bfloat16).view(2, P, asym.PAGE_TOKENS, 128)
        row = {"kv_MB": round(p.kv_bytes / 1e6, 1), "pool_pages": P,
               "map_agree": f"{info['verify_agree']}/{info['verify_classified']}"}
        for where, xm in (("chip", 0), ("one_die", g0)):
            plan = asym.attn_decode_plan(B, 32, 8, S, topo=topo, xcd_mask=xm)
            tabs = {}
            for name, pol in (("in_order", asym.PAGES_IN_ORDER), ("local", asym.PAGES_LOCAL),
                              ("remote", asym.PAGES_REMOTE)):
                kt = asym.attn_pages_place(plan, B, 8, S, P, pol, homes[:P], grp)
                vt = asym.attn_pages_place(plan, B, 8, S, P, pol, homes[P:], grp)
                tabs[name] = (torch.as_tensor(kt).to(dev), torch.as_tensor(vt).to(dev))
            fns = {"dense": lambda: asym.attn_decode(q, k, v, topo=topo, xcd_mask=xm)}
            outs = {}
            for name, (kt, vt) in tabs.items():
                pools[0].copy_(workloads.page_pool(k, kt, P))
                pools[1].copy_(workloads.page_pool(v, vt, P))
                o = asym.attn_decode_paged(q, pools[0], pools[1], kt, vt, S, topo=topo, xcd_mask=xm)
                fns_one = {name: lambda kt=kt, vt=vt: asym.attn_decode_paged(q, pools[0], pools[1], kt, vt, S,
                                                                              topo=topo, xcd_mask=xm)}
                outs[name] = queued(fns_one, launches, rounds, stream)[name]
                row.setdefault("bitwise_equal_to_dense", {})[f"{where}_{name}"] = bool(
                    torch.equal(o, asym.attn_decode(q, k, v, topo=topo, xcd_mask=xm)))
            outs["dense"] = queued(fns, launches, rounds, stream)["dense"]
            r = {k_: {"us": round(1e3 * ms, 2), "GBps": round(p.kv_bytes / (ms * 1e-3) / 1e9, 1)}
                 for k_, ms in outs.items()}
            r["local_over_remote"] = round(outs["remote"] / outs["local"], 3)
            r["local_over_in_order"] = round(outs["in_order"] / outs["local"], 3)
            r["local_over_dense"] = round(outs["dense"] / outs["local"], 3)
            row[where] = r
        out[f"B{B}_S{S}"] = row
        del raw, pools, q, k, v
        torch.cuda.empty_cache()
    return out


def attention_study(topo, dev, stream, masked: bool, launches: int = 5, rounds: int = 3):
    """Decode attention (32 query heads, head dimension 128; grouped-query with
    8 key/value heads and multi-head with 32) over batch and KV length: the
    logical KV working set W = 4 B S_k H_kv D bytes per time, aware and
    oblivious on the full GPU, and on one seeded random 128-CU set (unequal CUs
    per XCD) with the same attention running on the complementary CUs."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    out = {}
    for kind in ("gqa", "mha"):
        for B in (1, 16, 64):
            for S in (1024, 8192, 32768):
                p = workloads.attn_problem(kind, B, S)
                if p.kv_bytes > (16 << 30):
                    continue
                q, k, v = workloads.make_attn_inputs_on(p, dev)
                o = torch.empty_like(q)
                fns = {m: (lambda m=m: asym.attn_decode(q, k, v, o, mapping=m, stream=stream))
                       for m in ("aware", "oblivious_rowmajor")}
                for f in fns.values():
                    f()
                ms = queued(fns, launches, rounds, stream)
                out[p.name] = {"W_GB": round(p.kv_bytes / 1e9, 4),
                               **{f"{m}_us": round(1e3 * t, 2) for m, t in ms.items()},
                               "aware_TBps_W": round(p.kv_bytes / (ms["aware"] * 1e-3) / 1e12, 3)}
                del q, k, v, o
    torch.cuda.empty_cache()
    # unequal CU counts: a seeded random 128-CU set, the complement running the same work
    res = {}
    if masked:
        p = workloads.attn_problem("gqa", 16, 8192)
        q, k, v = workloads.make_attn_inputs_on(p, dev)
        q2, k2, v2 = workloads.make_attn_inputs_on(p, dev)
        o, o2 = torch.empty_like(q), torch.empty_like(q)
        mask = workloads.random_mask_bits(workloads.COLOC.seed, 1, 128)[0]
        comp = [b for b in range(256) if b not in set(mask)]
        sa, sb = asym.stream_create(topo, mask), asym.stream_create(topo, comp)
        try:
            for m in ("aware", "oblivious_rowmajor"):
                f = lambda: asym.attn_decode(q, k, v, o, mapping=m, topo=topo, stream=sa)
                g = lambda: asym.attn_decode(q2, k2, v2, o2, mapping="aware", topo=topo, stream=sb)
                for _ in range(3):
                    f(), g()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(sa)
                for _ in range(20):
                    f()
                    g()
                e1.record(sa)
                torch.cuda.synchronize()
                t = e0.elapsed_time(e1) / 20
                res[m] = {"us": round(1e3 * t, 2), "TBps_W": round(p.kv_bytes / (t * 1e-3) / 1e12, 3)}
            res["cus_per_xcd"] = topo.cuset_counts(mask)
            res["workload"] = p.name
        finally:
            asym.stream_destroy(sa)
            asym.stream_destroy(sb)
        del q, k, v, q2, k2, v2
        torch.cuda.empty_cache()
    return {"configs": out, "random_128_cu_set_with_tenant": res}


def mla_study(topo, dev, stream, masked: bool, launches: int = 5, rounds: int = 3):
    """Latent-attention decode (576-wide cache rows shared by all query heads):
    16 and 128 query heads over batch and KV length, W = 2 B S_k (512 + 64)
    bytes per time, aware and oblivious on the full GPU; then on CU sets with
    unequal counts: the two I/O dies at 28 and 32 CUs per XCD (the analog of
    the paper's 70/78-SM partitions), and a seeded random 128-CU set with the
    same attention on the complementary CUs."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    out = {}
    for Hq in (16, 128):
        for B in (1, 16, 64):
            for S in (4096, 32768):
                p = workloads.mla_problem(B, Hq, S)
                q, kv = workloads.make_mla_inputs_on(p, dev)
                o = torch.empty((B, Hq, 512), dtype=torch.bfloat16, device=dev)
                fns = {m: (lambda m=m: asym.mla_decode(q, kv, o, mapping=m, topo=topo, stream=stream))
                       for m in ("aware", "oblivious_rowmajor")}
                for f in fns.values():
                    f()
                ms = queued(fns, launches, rounds, stream)
                flops = 2.0 * B * Hq * S * (576 + 512)
                out[p.name] = {"W_GB": round(p.kv_bytes / 1e9, 4),
                               **{f"{m}_us": round(1e3 * t, 2) for m, t in ms.items()},
                               "aware_TBps_W": round(p.kv_bytes / (ms["aware"] * 1e-3) / 1e12, 3),
                               "aware_tflops": round(flops / (ms["aware"] * 1e-3) / 1e12, 1),
                               "speedup_vs_oblivious": round(ms["oblivious_rowmajor"] / ms["aware"], 4)}
                del q, kv, o
    torch.cuda.empty_cache()
    uneven = {}
    if masked:
        # die-uneven set: 4 CUs taken off each XCD of the first I/O die (28 / 32 CUs per XCD)
        g = topo.info()["group_of_xcd"]
        die0 = [x for x in range(8) if (g[x] == 0 if g and min(g) >= 0 else x < 4)]
        cus = topo.cus()
        drop, seen = set(), {x: 0 for x in die0}
        for c in cus:
            if c["xcc"] in seen and seen[c["xcc"]] < 4:
                drop.add(c["mask_bit"])
                seen[c["xcc"]] += 1
        die_mask = [c["mask_bit"] for c in cus if c["mask_bit"] not in drop]
        for name, (B, Hq, S) in (("B64_H128_S8192", (64, 128, 8192)), ("B16_H16_S32768", (16, 16, 32768))):
            p = workloads.mla_problem(B, Hq, S)
            q, kv = workloads.make_mla_inputs_on(p, dev)
            o = torch.empty((B, Hq, 512), dtype=torch.bfloat16, device=dev)
            s = asym.stream_create(topo, die_mask)
            try:
                fns = {m: (lambda m=m: asym.mla_decode(q, kv, o, mapping=m, topo=topo, stream=s))
                       for m in ("aware", "oblivious_rowmajor")}
                for f in fns.values():
                    f()
                ms = queued(fns, launches, rounds, s)
            finally:
                asym.stream_destroy(s)
            uneven[f"die_28_32_{name}"] = {"cus_per_xcd": topo.cuset_counts(die_mask),
                                           **{f"{m}_us": round(1e3 * t, 2) for m, t in ms.items()},
                                           "speedup_vs_oblivious": round(ms["oblivious_rowmajor"] / ms["aware"], 4)}
            del q, kv, o
        p = workloads.mla_problem(16, 128, 8192)
        q, kv = workloads.make_mla_inputs_on(p, dev)
        q2, kv2 = workloads.make_mla_inputs_on(p, dev)
        o, o2 = torch.empty((16, 128, 512), dtype=torch.bfloat16, device=dev), \
            torch.empty((16, 128, 512), dtype=torch.bfloat16, device=dev)
        mask = workloads.random_mask_bits(workloads.COLOC.seed, 1, 128)[0]
        comp = [b for b in range(256) if b not in set(mask)]
        sa, sb = asym.stream_create(topo, mask), asym.stream_create(topo, comp)
        res = {}
        try:
            for m in ("aware", "oblivious_rowmajor"):
                f = lambda: asym.mla_decode(q, kv, o, mapping=m, topo=topo, stream=sa)
                gg = lambda: asym.mla_decode(q2, kv2, o2, mapping="aware", topo=topo, stream=sb)
                for _ in range(3):
                    f(), gg()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(sa)
                for _ in range(10):
                    f()
                    gg()
                e1.record(sa)
                torch.cuda.synchronize()
                t = e0.elapsed_time(e1) / 10
                res[m] = {"us": round(1e3 * t, 2), "TBps_W": round(p.kv_bytes / (t * 1e-3) / 1e12, 3)}
            res["cus_per_xcd"] = topo.cuset_counts(mask)
            res["workload"] = p.name
        finally:
            asym.stream_destroy(sa)
            asym.stream_destroy(sb)
        uneven["random_128_cu_set_with_tenant"] = res
        del q, kv, q2, kv2, o, o2
        torch.cuda.empty_cache()
    return {"configs": out, "uneven_cu_sets": uneven}


FOCUS = ("decode_gemm", "grouped_small_m", "grouped_expert", "attention_gqa", "attention_b1", "chunk_read", "mla",
         "mla_long", "mla16", "copy", "gemm16k")


def focus_run(name: str, dev, stream, launches: int, mapping: str = "aware") -> dict:
    """One workload launched `launches` times after 3 warm-ups (for profiler runs):
      gemm16k          the persistent GEMM at 16384^3 (operands beyond the memory-side
                       cache), in `mapping` (--mapping-only; default aware)
      decode_gemm      small-M GEMM 32 x 14336 x 4096 (decode projection)
      grouped_small_m  grouped GEMM (32 groups of ~20 rows) x (6144, 7168), seed 5
      grouped_expert   grouped GEMM (6 groups of ~1024 rows) x (6144, 7168), seed 1, on
                       the persistent kernel, in `mapping`
      attention_gqa    decode attention, grouped-query, B = 64, S_k = 32768
      attention_b1     decode attention, grouped-query, B = 1, S_k = 32768 (latency-bound)
      chunk_read       strided read of a 16 GiB region in 8 KiB chunks, address order
      mla              latent-attention decode, B = 64, H_q = 128, S_k = 8192 (aware)
      mla_long         latent-attention decode, B = 64, H_q = 128, S_k = 32768 (aware)
      mla16            latent-attention decode, B = 64, H_q = 16, S_k = 32768 (aware)
      copy             the streaming copy, 64 MiB, one pass, whole chip
    Reports the mean per launch (HIP events on the launch stream) and the
    algorithmic bytes each launch must read or write."""
    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads
    if name == "decode_gemm":
        (_, _), (da, db) = workloads.make_pd_inputs()
        A, B = da.to(dev), db.to(dev)
        C = torch.empty((A.shape[0], B.shape[0]), dtype=torch.bfloat16, device=dev)
        fn = lambda: asym.gemm(A, B, C, stream=stream)
        nbytes = 2 * (A.numel() + B.numel() + C.numel())
        kernel = "gemm_bf16_small_m<2, 8>"
    elif name == "grouped_small_m":
        p = workloads.grouped_problem(32, 20, 6144, 7168)
        Ms, A, B = workloads.make_grouped_inputs_on(p, dev)
        C = torch.empty((sum(Ms), p.N), dtype=torch.bfloat16, device=dev)
        fn = lambda: asym.gemm_grouped(A, B, Ms, C, stream=stream)
        nbytes = p.working_set_bytes
        kernel = "gemm_bf16_small_m<2, 8>"
    elif name == "grouped_expert":
        p = workloads.grouped_problem(6, 1024, 6144, 7168, seed=1)
        Ms, A, B = workloads.make_grouped_inputs_on(p, dev)
        C = torch.empty((sum(Ms), p.N), dtype=torch.bfloat16, device=dev)
        fn = lambda: asym.gemm_grouped(A, B, Ms, C, mapping=mapping, stream=stream)
        nbytes = p.working_set_bytes
        kernel = f"gemm_bf16_persistent (grouped, {mapping})"
    elif name == "attention_gqa":
        p = workloads.attn_problem("gqa", 64, 32768)
        q, k, v = workloads.make_attn_inputs_on(p, dev)
        o = torch.empty_like(q)
        fn = lambda: asym.attn_decode(q, k, v, o, stream=stream)
        nbytes = p.kv_bytes + 2 * 2 * q.numel()
        kernel = "attn_decode_split<4, false> + attn_decode_merge"
    elif name == "attention_b1":
        p = workloads.attn_problem("gqa", 1, 32768)
        q, k, v = workloads.make_attn_inputs_on(p, dev)
        o = torch.empty_like(q)
        fn = lambda: asym.attn_decode(q, k, v, o, stream=stream)
        nbytes = p.kv_bytes + 2 * 2 * q.numel()
        kernel = "attn_decode_split<4, false> + attn_decode_merge"
    elif name in ("mla", "mla_long"):
        p = workloads.mla_problem(64, 128, 8192 if name == "mla" else 32768)
        q, kv = workloads.make_mla_inputs_on(p, dev)
        o = torch.empty((64, 128, 512), dtype=torch.bfloat16, device=dev)
        fn = lambda: asym.mla_decode(q, kv, o, stream=stream)
        nbytes = p.kv_bytes + 2 * q.numel() + 2 * o.numel()
        kernel = "mla_decode_split_wg<2> + mla_decode_merge"
    elif name == "mla16":
        p = workloads.mla_problem(64, 16, 32768)
        q, kv = workloads.make_mla_inputs_on(p, dev)
        o = torch.empty((64, 16, 512), dtype=torch.bfloat16, device=dev)
        fn = lambda: asym.mla_decode(q, kv, o, stream=stream)
        nbytes = p.kv_bytes + 2 * q.numel() + 2 * o.numel()
        kernel = "mla_decode_split + mla_decode_merge"
    elif name == "copy":
        src = workloads.copy_source(workloads.COPY_BYTES // 2).to(dev)
        dst = torch.empty_like(src)
        fn = lambda: asym.copy(dst, src, passes=1, stream=stream)
        nbytes = 2 * workloads.COPY_BYTES
        kernel = "copy_kernel"
    elif name == "gemm16k":
        n = 16384
        g = torch.Generator(device=dev).manual_seed(1)
        A = (torch.rand((n, n), generator=g, device=dev) * 2 - 1).to(torch.bfloat16)
        B = (torch.rand((n, n), generator=g, device=dev) * 2 - 1).to(torch.bfloat16)
        C = torch.empty((n, n), dtype=torch.bfloat16, device=dev)
        fn = lambda: asym.gemm(A, B, C, mapping=mapping, stream=stream)
        nbytes = 3 * 2 * n * n
        kernel = f"gemm_bf16_persistent<true, 8, 0, false> ({mapping})"
    elif name == "chunk_read":
        nb = 16 << 30
        raw = torch.empty(nb + (2 << 20), dtype=torch.uint8, device=dev)
        ptr = raw.data_ptr() + ((-raw.data_ptr()) % (2 << 20))
        raw.fill_(1)
        import numpy as np
        homes = np.zeros(nb >> 13, dtype=np.int8)
        chunks, off = asym.chunk_lists(homes, 8, [0] * 4 + [1] * 4, asym.CHUNKS_ALL)
        fn = lambda: asym.chunk_read_bw(ptr, nb, 13, chunks, off, iters=1, stream=stream)
        nbytes = nb
        kernel = "chunk_read_kernel"
    else:
        raise ValueError(name)
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    if name == "chunk_read":
        ms = sum(fn()[0] for _ in range(launches)) / launches
    else:
        ms = queued({"f": fn}, launches, 1, stream)["f"]
    if name == "gemm16k":
        return {"focus": name, "kernel": kernel, "launches": launches, "ms_per_launch": round(ms, 5),
                "tflops": round(2.0 * 16384 ** 3 / (ms * 1e-3) / 1e12, 1), "compulsory_bytes": int(nbytes)}
    return {"focus": name, "kernel": kernel, "launches": launches, "ms_per_launch": round(ms, 5),
            "algorithmic_bytes": int(nbytes), "TBps": round(nbytes / (ms * 1e-3) / 1e12, 3)}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--settle", type=float, default=2.0,
                    help="seconds of untimed launches before timing (clock and power settle)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-rows", type=int, default=8192,
                    help="rows of A in the CPU oracle sample (8192 = the whole problem)")
    ap.add_argument("--probe", choices=("full", "maskmap", "identity"), default="full",
                    help="topology probe run first: full = identity, mask map and the per-XCD "
                         "latency / affinity probe; profiling runs use 'identity' (the profiler's "
                         "queue interception does not survive CU-masked stream creation)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy 10 times (scale for byte counters)")
    ap.add_argument("--studies", default="compare,grid,large,llm,pd,pd_trace,spread,balanced,grouped,numa,placed,attention,mla,parity",
                    help="comma list of extra studies: compare (interleaved mappings at 8192^3), "
                         "grid (tile-column counts not multiples of 8), large (operands beyond the "
                         "memory-side cache, 12288^3 to 16384^3), llm (decoder shapes), pd (prefill || decode), spread (128-CU sets), "
                         "grouped (expert-layer grouped GEMMs), numa (partition hash and local / "
                         "remote read bandwidth), attention (decode attention), mla (latent-"
                         "attention decode), parity (every "
                         "configuration's product against the oracle, all outputs); 'none' for "
                         "the headline only")
    ap.add_argument("--spread-masks", type=int, default=32)
    ap.add_argument("--spread-tenants", default="copy",
                    help="comma list of tenants for the CU-set spread study: copy (the 64 MiB "
                         "streaming copy), gemm (a second GEMM), read (a whole-buffer reader)")
    ap.add_argument("--spread-repeats", type=int, default=5)
    ap.add_argument("--focus", choices=FOCUS, default=None,
                    help="run only this workload (profiling runs); prints its own JSON line")
    ap.add_argument("--mapping-only", default=None,
                    help="time only this mapping, no studies (profiling runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "the GEMM would shard by output columns with no exchange, see the design notes",
              file=sys.stderr)
        return 2

    import torch

    import paper_2609_24270_amd as asym
    from paper_2609_24270_amd import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    asym.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        src = torch.ones(128 << 20, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_each_way": src.numel() * 2, "launches": 10}))
        return 0
    if args.focus:
        print(json.dumps(focus_run(args.focus, dev, torch.cuda.current_stream(), args.steps,
                                   args.mapping_only or "aware")), flush=True)
        return 0
    studies = set() if args.mapping_only or args.studies == "none" else set(args.studies.split(","))
    if args.probe == "identity":
        studies -= {"pd", "pd_trace", "spread", "balanced"}  # CU-masked sets need the mask map
    p = workloads.SQUARE_8192
    A, B = workloads.make_inputs(p)
    Ad, Bd = A.to(dev), B.to(dev)
    C = torch.empty((p.M, p.N), dtype=torch.bfloat16, device=dev)
    t0 = time.perf_counter()
    flags = asym.PROBE_IDENTITY
    if args.probe in ("full", "maskmap"):
        flags |= asym.PROBE_MASKMAP
    if args.probe == "full":
        flags |= asym.PROBE_LATENCY
    topo = asym.probe_topology(0, flags)
    probe_s = time.perf_counter() - t0
    info = topo.info()
    halves = affinity_halves(topo, info["n_xcds"])
    stream = torch.cuda.current_stream()

    head_mapping = args.mapping_only or "aware"
    fns = {m: (lambda m=m: asym.gemm(Ad, Bd, C, mapping=m, topo=topo, stream=stream)) for m in MAPPINGS}
    head = fns[head_mapping]
    plan = asym.gemm_plan(Ad, Bd, C, mapping=head_mapping, topo=topo, stream=stream)
    for _ in range(args.warmup):
        head()
    dinfo = asym.device_query(0)
    sampler = ClockPowerSampler(dinfo["pci_bus_id"])
    with sampler:
        settle([head], args.settle)
        total_ms, per_launch_ms = time_launches(head, args.steps, stream)
    ms_per_step = total_ms / args.steps
    tflops = p.flops / (ms_per_step * 1e-3) / 1e12
    achieved = p.flops / (per_launch_ms * 1e-3) / 1e12

    line = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "square bf16 GEMM M=N=K=8192, uniform[-1,1] seed 1, B [N,K], "
                               f"full GPU, {head_mapping} persistent mapping, topology probe first",
                   "M": p.M, "N": p.N, "K": p.K, "mapping": head_mapping, "plan": plan},
        "pct_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 2),
        "clock_power": clock_power(sampler.summary(), achieved),
        "device": {k: dinfo[k] for k in ("arch", "pci_bus_id", "compute_partition", "memory_partition")},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic()},
        "topology": {"cus_per_xcd": info["cus_per_xcd"], "probe_s": round(probe_s, 3),
                     "round_robin_dispatch": topo.dispatch_rr_fraction(),
                     "affinity": affinity_summary(topo) if args.probe == "full" else None},
    }
    if "compare" in studies:
        ms = interleaved(fns, args.steps, stream)
        line["mappings_interleaved"] = {m: {"per_launch_ms": round(ms[m], 5),
                                            "tflops": round(p.flops / (ms[m] * 1e-3) / 1e12, 2)}
                                        for m in MAPPINGS}
        line["aware_speedup_vs_oblivious_grouped"] = round(ms["oblivious_grouped"] / ms["aware"], 4)
        line["aware_speedup_vs_oblivious_rowmajor"] = round(ms["oblivious_rowmajor"] / ms["aware"], 4)
        # context: the vendor library on the same operands (not the product path)
        Bt = Bd.t().contiguous()
        mm = lambda: torch.mm(Ad, Bt)
        settle([mm], 0.3)
        tot, per = time_launches(mm, 10, stream)
        line["context"] = {"torch_matmul_tflops": round(p.flops / (tot / 10 * 1e-3) / 1e12, 2)}
        del Bt
    if "grid" in studies:
        line["tile_grid_shapes"] = grid_study(topo, dev, stream)
    if "large" in studies:
        line["beyond_mall_shapes"] = large_study(topo, dev, stream)
    if "llm" in studies:
        line["square_512"] = square_512(topo, dev, stream)
        line["llm_shapes_tflops"] = llm_shapes(dev, stream, 20)
        line["decode_gemm"] = decode_gemm(dev, stream)
        line["decode_projections"] = decode_projections(dev, stream)
    if "pd" in studies:
        line["prefill_decode"] = prefill_decode(topo, dev, 10, halves, warm=100)
        line["prefill_decode_after_idle"] = prefill_decode(topo, dev, 10, halves, warm=0)
    if "pd_trace" in studies:
        line["prefill_trace"] = pd_trace(topo, dev, halves)
    if "spread" in studies:
        for tenant in args.spread_tenants.split(","):
            key = "cu_set_spread" if tenant == "copy" else f"cu_set_spread_{tenant}_tenant"
            line[key] = spread_study(topo, dev, args.spread_masks, 20, halves, tenant, args.spread_repeats)
    if "balanced" in studies:
        line["balanced_sets"] = balanced_study(topo, dev)
    if "grouped" in studies:
        line["grouped_gemm"] = grouped_study(dev, stream, range(1, 6), 8, 5)
    if "attention" in studies:
        line["decode_attention"] = attention_study(topo, dev, stream, args.probe != "identity")
    if "mla" in studies:
        line["mla_decode"] = mla_study(topo, dev, stream, args.probe != "identity")
    if "numa" in studies or "placed" in studies:
        summ, hres = interleave_summary(dev)
        line["partition_hash"] = summ
        if hres["n_groups"] == 2 and "numa" in studies:
            line["numa_read_bw"] = numa_bw_study(dev, hres)
        if hres["n_groups"] == 2 and "placed" in studies:
            line["placed_attention"] = placed_attention_study(dev, hres, topo, stream)
    if args.no_cpu:
        line["cpu_baseline"] = None
    else:
        # the timed problem once more, so C holds the head mapping's output
        head()
        torch.cuda.synchronize()
        cpu, parity = cpu_baseline(A, B, args.cpu_rows, C.cpu())
        line["cpu_baseline"] = {k: (round(v, 6) if isinstance(v, float) else v) for k, v in cpu.items()}
        line["parity_vs_oracle"] = parity
        if args.probe != "identity" and "parity" in studies:
            line["config_parity"] = config_parity(topo, dev, stream)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
