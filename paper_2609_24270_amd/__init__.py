"""asym: asymmetry-aware persistent bf16 GEMM scheduling for MI355X (gfx950).

Thin ctypes binding of libasym.so (C ABI in include/asym.h).  Every step of
the hot path runs in the library's HIP kernels; this module only marshals
arguments (tensor data pointers, stream handles, host arrays).  PyTorch is used
for device memory and streams.  There is no fallback: if libasym.so is missing
or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import json
import os
from typing import Optional, Sequence

from . import workloads  # noqa: F401  (seeded inputs; no method arithmetic)

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libasym.so")

MASK_WORDS = 8
MAX_XCDS = 16
MAX_CUS = MASK_WORDS * 32

OK, EINVAL, EHIP, EUNSUPPORTED, ETIMEOUT, EINVARIANT, ENOMEM, ENOCACHE = 0, -1, -2, -3, -4, -5, -6, -7
MAP_AWARE, MAP_OBLIVIOUS_GROUPED, MAP_OBLIVIOUS_ROWMAJOR = 0, 1, 2
MAPPINGS = {"aware": MAP_AWARE, "oblivious_grouped": MAP_OBLIVIOUS_GROUPED,
            "oblivious_rowmajor": MAP_OBLIVIOUS_ROWMAJOR}
B_NK, B_KN = 0, 1
PROBE_IDENTITY, PROBE_MASKMAP, PROBE_LATENCY = 1, 2, 4
CUSET_XCD_ALIGNED, CUSET_AFFINITY_ALIGNED, CUSET_STRIPED, CUSET_RANDOM = 0, 1, 2, 3

# Every function the C ABI exports (include/asym.h), in declaration order.
EXPORTS = (
    "asym_device_query", "asym_topology_cache_key", "asym_probe_topology",
    "asym_topology_save", "asym_topology_load", "asym_topology_from_records",
    "asym_topology_free", "asym_topology_info", "asym_topology_cu",
    "asym_topology_dispatch", "asym_topology_latency", "asym_topology_json",
    "asym_latency_params_default", "asym_latency_probe", "asym_latency_analyze",
    "asym_interleave_params_default", "asym_interleave_probe", "asym_interleave_analyze",
    "asym_home_map", "asym_home_map_analyze", "asym_chunk_lists", "asym_chunk_read_bw", "asym_chunk_read",
    "asym_dispatch_check", "asym_dispatch_probe", "asym_cuset_split_xcds",
    "asym_cuset_make", "asym_cuset_counts", "asym_stream_create",
    "asym_stream_destroy", "asym_schedule_build", "asym_grouped_schedule_build",
    "asym_gemm_bf16", "asym_gemm_grouped_bf16", "asym_gemm_bf16_noalloc", "asym_gemm_noalloc_limits",
    "asym_gemm_bf16_trace",
    "asym_gemm_plan", "asym_gemm_set_small_m",
    "asym_attn_decode_bf16", "asym_attn_decode_plan", "asym_attn_decode_paged_bf16", "asym_attn_pages_place", "asym_mla_decode_bf16", "asym_mla_decode_plan", "asym_mla_set_workgroup_form",
    "asym_copy_bf16", "asym_corun", "asym_last_error", "asym_version",
)


class AsymError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"asym error {status}: {msg}")
        self.status = status


class DeviceInfo(ctypes.Structure):
    _fields_ = [("n_cus", ctypes.c_int), ("n_xccs", ctypes.c_int),
                ("n_cus_physical", ctypes.c_int), ("clock_khz", ctypes.c_int),
                ("wall_clock_khz", ctypes.c_int), ("lds_bytes_per_cu", ctypes.c_int),
                ("l2_bytes", ctypes.c_int), ("hbm_bytes", ctypes.c_size_t),
                ("arch", ctypes.c_char * 64), ("pci_bus_id", ctypes.c_char * 32),
                ("uuid", ctypes.c_char * 40), ("runtime_version", ctypes.c_int),
                ("driver_version", ctypes.c_int), ("compute_partition", ctypes.c_char * 16),
                ("memory_partition", ctypes.c_char * 16)]


class LatencyParams(ctypes.Structure):
    _fields_ = [("alloc_bytes", ctypes.c_size_t), ("n_samples", ctypes.c_int),
                ("passes", ctypes.c_int), ("l2_samples", ctypes.c_int),
                ("seed", ctypes.c_uint64), ("group_threshold", ctypes.c_double),
                ("tie_cycles", ctypes.c_double)]


class LatencySummary(ctypes.Structure):
    _fields_ = [("n_xcds", ctypes.c_int), ("n_samples", ctypes.c_int),
                ("passes", ctypes.c_int), ("l2_samples", ctypes.c_int),
                ("timer_overhead", ctypes.c_double), ("clock_mhz", ctypes.c_double),
                ("l2_hit", ctypes.c_double * MAX_XCDS),
                ("mall_hit", ctypes.c_double * MAX_XCDS),
                ("hbm", ctypes.c_double * MAX_XCDS),
                ("group_of_xcd", ctypes.c_int * MAX_XCDS),
                ("n_groups", ctypes.c_int),
                ("home_share", ctypes.c_double * MAX_XCDS),
                ("unclassified_share", ctypes.c_double),
                ("corr", (ctypes.c_double * MAX_XCDS) * MAX_XCDS),
                ("hbm_by_home", (ctypes.c_double * MAX_XCDS) * MAX_XCDS)]

    def to_dict(self) -> dict:
        nx, ng = self.n_xcds, self.n_groups
        return {"n_xcds": nx, "n_samples": self.n_samples, "passes": self.passes,
                "l2_samples": self.l2_samples, "timer_overhead": self.timer_overhead,
                "clock_mhz": self.clock_mhz, "l2_hit": list(self.l2_hit)[:nx],
                "mall_hit": list(self.mall_hit)[:nx], "hbm": list(self.hbm)[:nx],
                "group_of_xcd": list(self.group_of_xcd)[:nx], "n_groups": ng,
                "home_share": list(self.home_share)[:ng],
                "unclassified_share": self.unclassified_share,
                "corr": [list(self.corr[x])[:nx] for x in range(nx)],
                "hbm_by_home": [list(self.hbm_by_home[x])[:ng] for x in range(nx)]}


class InterleaveParams(ctypes.Structure):
    _fields_ = [("n_bases", ctypes.c_int), ("lo_bit", ctypes.c_int), ("hi_bit", ctypes.c_int),
                ("n_pairs", ctypes.c_int), ("passes", ctypes.c_int), ("seed", ctypes.c_uint64),
                ("group_threshold", ctypes.c_double), ("tie_cycles", ctypes.c_double),
                ("decide", ctypes.c_double)]


class InterleaveResult(ctypes.Structure):
    _fields_ = [("n_xcds", ctypes.c_int), ("n_groups", ctypes.c_int),
                ("group_of_xcd", ctypes.c_int * MAX_XCDS), ("n_addresses", ctypes.c_int),
                ("block", ctypes.c_int), ("flip_fraction", ctypes.c_double * 64),
                ("usable", ctypes.c_int * 64), ("verdict", ctypes.c_int * 64),
                ("hash_mask", ctypes.c_uint64), ("lowest_bit", ctypes.c_int),
                ("determined_below", ctypes.c_int), ("granularity", ctypes.c_int64),
                ("pair_checks", ctypes.c_int), ("pair_agree", ctypes.c_int),
                ("linear_consistency", ctypes.c_double), ("unclassified_share", ctypes.c_double),
                ("local_cycles", ctypes.c_double), ("remote_cycles", ctypes.c_double),
                ("base_align", ctypes.c_uint64)]

    def to_dict(self) -> dict:
        d = {k: getattr(self, k) for k, _ in self._fields_
             if k not in ("group_of_xcd", "flip_fraction", "usable", "verdict")}
        d["group_of_xcd"] = list(self.group_of_xcd)[:self.n_xcds]
        d["flip_fraction"] = list(self.flip_fraction)
        d["usable"] = list(self.usable)
        d["verdict"] = list(self.verdict)
        return d


class HomeMapInfo(ctypes.Structure):
    _fields_ = [("n_pages", ctypes.c_int), ("n_chunks", ctypes.c_int), ("n_groups", ctypes.c_int),
                ("group_of_xcd", ctypes.c_int * MAX_XCDS), ("unclassified_pages", ctypes.c_int),
                ("chunk_share", ctypes.c_double * 2), ("n_verify", ctypes.c_int),
                ("verify_classified", ctypes.c_int), ("verify_agree", ctypes.c_int),
                ("local_cycles", ctypes.c_double), ("remote_cycles", ctypes.c_double)]

    def to_dict(self, n_xcds: int) -> dict:
        d = {k: getattr(self, k) for k, _ in self._fields_ if k not in ("group_of_xcd", "chunk_share")}
        d["group_of_xcd"] = list(self.group_of_xcd)[:n_xcds]
        d["chunk_share"] = list(self.chunk_share)
        return d


CHUNKS_ALL, CHUNKS_LOCAL, CHUNKS_REMOTE = 0, 1, 2


class Task(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("mask", ctypes.c_uint32 * MASK_WORDS),
                ("xcd_mask", ctypes.c_uint32), ("iters", ctypes.c_int),
                ("mapping", ctypes.c_int), ("M", ctypes.c_int), ("N", ctypes.c_int),
                ("K", ctypes.c_int), ("A", ctypes.c_void_p), ("B", ctypes.c_void_p),
                ("C", ctypes.c_void_p), ("src", ctypes.c_void_p), ("dst", ctypes.c_void_p),
                ("n_bytes", ctypes.c_size_t), ("grid", ctypes.c_int), ("warm_iters", ctypes.c_int)]


class MlaPlanInfo(ctypes.Structure):
    _fields_ = [("split_tokens", ctypes.c_int), ("n_splits", ctypes.c_int), ("head_blocks", ctypes.c_int),
                ("tasks", ctypes.c_int), ("grid", ctypes.c_int), ("tasks_per_workgroup", ctypes.c_int),
                ("n_xcds", ctypes.c_int), ("tasks_per_xcd", ctypes.c_int * MAX_XCDS),
                ("workgroup_form", ctypes.c_int), ("workspace_bytes", ctypes.c_size_t),
                ("static_deal", ctypes.c_int)]

    def to_dict(self) -> dict:
        d = {k: getattr(self, k) for k, _ in self._fields_ if k != "tasks_per_xcd"}
        d["tasks_per_xcd"] = list(self.tasks_per_xcd)[:self.n_xcds]
        return d


class GemmPlanInfo(ctypes.Structure):
    _fields_ = [("tile_m", ctypes.c_int), ("tile_n", ctypes.c_int),
                ("tiles_m", ctypes.c_int), ("tiles_n", ctypes.c_int),
                ("grid", ctypes.c_int), ("workers", ctypes.c_int),
                ("claims", ctypes.c_int), ("vector_path", ctypes.c_int),
                ("n_xcds", ctypes.c_int), ("workers_per_xcd", ctypes.c_int * MAX_XCDS),
                ("small_m", ctypes.c_int), ("k_splits", ctypes.c_int),
                ("b_transposed", ctypes.c_int)]

    def to_dict(self) -> dict:
        d = {k: getattr(self, k) for k, _ in self._fields_ if k != "workers_per_xcd"}
        d["workers_per_xcd"] = list(self.workers_per_xcd)[:self.n_xcds]
        return d


class AttnPlanInfo(ctypes.Structure):
    _fields_ = [("split_tokens", ctypes.c_int), ("n_splits", ctypes.c_int), ("tasks", ctypes.c_int),
                ("grid", ctypes.c_int), ("tasks_per_workgroup", ctypes.c_int), ("n_xcds", ctypes.c_int),
                ("tasks_per_xcd", ctypes.c_int * MAX_XCDS), ("workspace_bytes", ctypes.c_size_t),
                ("dense_static", ctypes.c_int)]

    def to_dict(self) -> dict:
        d = {k: getattr(self, k) for k, _ in self._fields_ if k != "tasks_per_xcd"}
        d["tasks_per_xcd"] = list(self.tasks_per_xcd)[:self.n_xcds]
        return d


class TaskResult(ctypes.Structure):
    _fields_ = [("ms_total", ctypes.c_double), ("ms_per_iter", ctypes.c_double),
                ("tflops", ctypes.c_double), ("gbps", ctypes.c_double),
                ("iters_done", ctypes.c_int), ("checksum", ctypes.c_uint32 * 4)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libasym.so and declare its signatures; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise AsymError(EUNSUPPORTED, f"{path} is not built; run paper_2609_24270_amd.build")
    lib = ctypes.CDLL(path)
    i, u32, vp, cp = ctypes.c_int, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_char_p
    ip = ctypes.POINTER(ctypes.c_int)
    u32p = ctypes.POINTER(ctypes.c_uint32)
    topo_p = ctypes.c_void_p
    sig = {
        "asym_device_query": (i, [i, ctypes.POINTER(DeviceInfo)]),
        "asym_topology_cache_key": (i, [i, cp, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)]),
        "asym_probe_topology": (i, [i, ctypes.c_uint, cp, ctypes.POINTER(topo_p)]),
        "asym_topology_save": (i, [topo_p, cp, cp]),
        "asym_topology_load": (i, [cp, cp, ctypes.c_uint, ctypes.POINTER(topo_p)]),
        "asym_topology_from_records": (i, [ctypes.POINTER(ctypes.c_int32), i, i, i,
                                           ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(topo_p)]),
        "asym_topology_free": (None, [topo_p]),
        "asym_topology_info": (i, [topo_p, ip, ip, ip, ip]),
        "asym_topology_cu": (i, [topo_p, i, ip, ip, ip, ip, ip]),
        "asym_topology_dispatch": (i, [topo_p, ctypes.POINTER(ctypes.c_double)]),
        "asym_topology_latency": (i, [topo_p, ctypes.POINTER(LatencySummary)]),
        "asym_latency_params_default": (None, [ctypes.POINTER(LatencyParams)]),
        "asym_dispatch_check": (i, [topo_p, u32p, ctypes.POINTER(ctypes.c_double), ip]),
        "asym_dispatch_probe": (i, [topo_p, u32p, i, ctypes.POINTER(ctypes.c_double), ip, ip]),
        "asym_cuset_split_xcds": (i, [topo_p, u32, u32p, u32p]),
        "asym_latency_probe": (i, [i, ctypes.POINTER(LatencyParams), u32p, ctypes.POINTER(LatencySummary)]),
        "asym_latency_analyze": (i, [u32p, i, i, ctypes.c_double, ctypes.c_double,
                                     ctypes.POINTER(LatencySummary)]),
        "asym_interleave_params_default": (None, [ctypes.POINTER(InterleaveParams)]),
        "asym_interleave_probe": (i, [i, ctypes.POINTER(InterleaveParams), ctypes.POINTER(ctypes.c_uint64),
                                      u32p, ctypes.POINTER(ctypes.c_int8), ctypes.POINTER(InterleaveResult)]),
        "asym_interleave_analyze": (i, [u32p, i, i, ctypes.POINTER(ctypes.c_uint64), i, ctypes.c_double,
                                        ctypes.c_double, ctypes.c_double, ctypes.POINTER(ctypes.c_int8),
                                        ctypes.POINTER(InterleaveResult)]),
        "asym_home_map": (i, [i, vp, ctypes.c_size_t, ctypes.c_uint64, i, ip, i, i, ctypes.c_uint64,
                              ctypes.c_double, ctypes.POINTER(ctypes.c_int8), ctypes.POINTER(HomeMapInfo)]),
        "asym_home_map_analyze": (i, [u32p, i, i, ctypes.POINTER(ctypes.c_uint64), i, ip, ctypes.c_uint64, i,
                                      ctypes.c_double, ctypes.POINTER(ctypes.c_int8),
                                      ctypes.POINTER(HomeMapInfo)]),
        "asym_chunk_lists": (i, [ctypes.POINTER(ctypes.c_int8), i, i, ip, u32, i, u32p, ip, ip]),
        "asym_chunk_read_bw": (i, [vp, ctypes.c_size_t, i, u32p, ip, i, i, vp, u32p,
                                   ctypes.POINTER(ctypes.c_double)]),
        "asym_chunk_read": (i, [vp, ctypes.c_size_t, i, u32p, ip, i, i, i, vp, u32p,
                                ctypes.POINTER(ctypes.c_double)]),
        "asym_topology_json": (i, [topo_p, cp, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)]),
        "asym_cuset_make": (i, [topo_p, i, i, ctypes.c_uint64, u32p, u32p]),
        "asym_cuset_counts": (i, [topo_p, u32p, ip]),
        "asym_stream_create": (i, [topo_p, u32p, ctypes.POINTER(vp)]),
        "asym_stream_destroy": (i, [vp]),
        "asym_schedule_build": (i, [i, i, i, ip, i, i, ip, ip, ip]),
        "asym_gemm_bf16": (i, [topo_p, i, i, i, vp, i, vp, i, i, vp, i, i, u32, vp]),
        "asym_grouped_schedule_build": (i, [i, ip, i, i, ip, i, ip, ip, ip]),
        "asym_gemm_grouped_bf16": (i, [topo_p, i, ip, i, i, vp, i, vp, i, vp, i, i, u32, vp]),
        "asym_gemm_plan": (i, [topo_p, i, i, i, vp, i, vp, i, i, vp, i, i, u32, vp,
                               ctypes.POINTER(GemmPlanInfo)]),
        "asym_gemm_set_small_m": (i, [i]),
        "asym_mla_set_workgroup_form": (i, [i]),
        "asym_gemm_bf16_noalloc": (i, [topo_p, i, i, i, vp, i, vp, i, i, vp, i, i, u32, vp]),
        "asym_gemm_bf16_trace": (i, [topo_p, i, i, i, vp, i, vp, i, i, vp, i, i, u32, vp, vp, i, ip]),
        "asym_gemm_noalloc_limits": (i, [ctypes.POINTER(ctypes.c_size_t), ip, ctypes.POINTER(ctypes.c_size_t)]),
        "asym_attn_decode_bf16": (i, [topo_p, i, i, i, i, i, vp, vp, vp, vp, vp, ctypes.c_float, i, i, u32, vp]),
        "asym_attn_decode_plan": (i, [topo_p, i, i, i, i, i, i, i, u32, vp, ctypes.POINTER(AttnPlanInfo)]),
        "asym_attn_decode_paged_bf16": (i, [topo_p, i, i, i, i, vp, vp, vp, ctypes.c_size_t, vp, vp, vp, vp,
                                            ctypes.c_float, i, i, u32, vp]),
        "asym_attn_pages_place": (i, [ctypes.POINTER(AttnPlanInfo), i, i, i, ctypes.POINTER(ctypes.c_int8),
                                      ctypes.c_size_t, ip, i, ctypes.POINTER(ctypes.c_int32)]),
        "asym_mla_decode_bf16": (i, [topo_p, i, i, i, vp, vp, vp, vp, ctypes.c_float, i, i, u32, vp]),
        "asym_mla_decode_plan": (i, [topo_p, i, i, i, i, i, u32, vp, ctypes.POINTER(MlaPlanInfo)]),
        "asym_copy_bf16": (i, [topo_p, vp, vp, ctypes.c_size_t, i, vp, u32, vp]),
        "asym_corun": (i, [topo_p, ctypes.POINTER(Task), i, ctypes.POINTER(TaskResult)]),
        "asym_last_error": (cp, []),
        "asym_version": (i, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(rc: int):
    if rc != OK:
        msg = load_library().asym_last_error()
        raise AsymError(rc, msg.decode() if msg else "")


def _ints(vals: Sequence[int]):
    arr = (ctypes.c_int * max(1, len(vals)))(*vals)
    return arr


def mask_words(bits: Optional[Sequence[int]]):
    """CU-mask bit positions -> ctypes uint32[8] (None -> None)."""
    if bits is None:
        return None
    m = (ctypes.c_uint32 * MASK_WORDS)()
    for b in bits:
        if not 0 <= b < MAX_CUS:
            raise ValueError(f"mask bit {b} out of range")
        m[b >> 5] |= 1 << (b & 31)
    return m


def mask_bits(words) -> list:
    return [w * 32 + b for w in range(MASK_WORDS) for b in range(32) if (words[w] >> b) & 1]


# ---- device -----------------------------------------------------------------

def device_query(device: int = 0) -> dict:
    info = DeviceInfo()
    _check(load_library().asym_device_query(device, ctypes.byref(info)))
    d = {k: getattr(info, k) for k, _ in DeviceInfo._fields_}
    for k in ("arch", "pci_bus_id", "uuid", "compute_partition", "memory_partition"):
        d[k] = getattr(info, k).decode()
    return d


def topology_cache_key(device: int = 0) -> str:
    """The key probe results of `device` are cached under (chip and mode)."""
    lib = load_library()
    need = ctypes.c_size_t()
    lib.asym_topology_cache_key(device, None, 0, ctypes.byref(need))
    buf = ctypes.create_string_buffer(max(1, need.value))
    _check(lib.asym_topology_cache_key(device, buf, need.value, ctypes.byref(need)))
    return buf.value.decode()


# ---- topology -----------------------------------------------------------

class Topology:
    """A probed (or record-built) topology map; owns the library object."""

    def __init__(self, handle: int):
        self._h = ctypes.c_void_p(handle)

    @property
    def handle(self):
        return self._h

    def __del__(self):
        if getattr(self, "_h", None) and self._h.value and _lib is not None:
            _lib.asym_topology_free(self._h)
            self._h = ctypes.c_void_p(0)

    def info(self) -> dict:
        n_cus, n_xcds = ctypes.c_int(), ctypes.c_int()
        per = (ctypes.c_int * MAX_XCDS)()
        grp = (ctypes.c_int * MAX_XCDS)()
        _check(load_library().asym_topology_info(self._h, ctypes.byref(n_cus), ctypes.byref(n_xcds), per, grp))
        nx = n_xcds.value
        return {"n_cus": n_cus.value, "n_xcds": nx, "cus_per_xcd": list(per)[:nx],
                "group_of_xcd": list(grp)[:nx]}

    def cu(self, idx: int) -> dict:
        vals = [ctypes.c_int() for _ in range(5)]
        _check(load_library().asym_topology_cu(self._h, idx, *[ctypes.byref(v) for v in vals]))
        return dict(zip(("xcc", "se", "sh", "cu", "mask_bit"), (v.value for v in vals)))

    def cus(self) -> list:
        return [self.cu(i) for i in range(self.info()["n_cus"])]

    def dispatch_rr_fraction(self) -> float:
        v = ctypes.c_double()
        _check(load_library().asym_topology_dispatch(self._h, ctypes.byref(v)))
        return v.value

    def latency(self) -> dict:
        s = LatencySummary()
        _check(load_library().asym_topology_latency(self._h, ctypes.byref(s)))
        return s.to_dict()

    def json(self) -> dict:
        lib = load_library()
        need = ctypes.c_size_t()
        lib.asym_topology_json(self._h, None, 0, ctypes.byref(need))
        buf = ctypes.create_string_buffer(need.value)
        _check(lib.asym_topology_json(self._h, buf, need.value, ctypes.byref(need)))
        return json.loads(buf.value.decode())

    def dispatch_check(self, mask: Optional[Sequence[int]] = None):
        """(share of workgroups on their residue class's XCC, workgroups per XCD)
        for a launch on the CU set `mask` (None = all CUs)."""
        rr = ctypes.c_double()
        per = (ctypes.c_int * MAX_XCDS)()
        _check(load_library().asym_dispatch_check(self._h, mask_words(mask), ctypes.byref(rr), per))
        return rr.value, list(per)[: self.info()["n_xcds"]]

    def dispatch_probe(self, pre_blocks: int = 0, mask: Optional[Sequence[int]] = None):
        """(class share, rotation, workgroups per XCD) of a launch right after a
        launch of pre_blocks workgroups on the same stream."""
        cf = ctypes.c_double()
        rot = ctypes.c_int()
        per = (ctypes.c_int * MAX_XCDS)()
        _check(load_library().asym_dispatch_probe(self._h, mask_words(mask), pre_blocks, ctypes.byref(cf),
                                                  ctypes.byref(rot), per))
        return cf.value, rot.value, list(per)[: self.info()["n_xcds"]]

    def cuset(self, n_cus: int, policy: int, seed: int = 0, exclude: Optional[Sequence[int]] = None) -> list:
        out = (ctypes.c_uint32 * MASK_WORDS)()
        _check(load_library().asym_cuset_make(self._h, n_cus, policy, seed, mask_words(exclude), out))
        return mask_bits(out)

    def cuset_split_xcds(self, xcd_mask_a: int):
        """(bits of side A, bits of side B): A works on the XCDs in xcd_mask_a,
        B on the rest; each side lends the other one CU per XCD."""
        a = (ctypes.c_uint32 * MASK_WORDS)()
        b = (ctypes.c_uint32 * MASK_WORDS)()
        _check(load_library().asym_cuset_split_xcds(self._h, xcd_mask_a, a, b))
        return mask_bits(a), mask_bits(b)

    def save(self, path: str, key: Optional[str] = None) -> None:
        """Write the map to a cache file (key: override the probe's own)."""
        _check(load_library().asym_topology_save(self._h, path.encode(), key.encode() if key else None))

    def cuset_counts(self, bits: Sequence[int]) -> list:
        per = (ctypes.c_int * MAX_XCDS)()
        _check(load_library().asym_cuset_counts(self._h, mask_words(bits), per))
        return list(per)[: self.info()["n_xcds"]]


def probe_topology(device: int = 0, flags: int = PROBE_IDENTITY, cache_path: Optional[str] = None) -> Topology:
    """Probe `device` (or reuse the map in cache_path when it was made on this
    chip and configuration with at least these probes; else probe and write it)."""
    h = ctypes.c_void_p()
    _check(load_library().asym_probe_topology(device, flags, cache_path.encode() if cache_path else None,
                                              ctypes.byref(h)))
    return Topology(h.value)


def topology_load(path: str, key: str, flags: int = PROBE_IDENTITY) -> Topology:
    """A map from a cache file, if made under `key` with at least `flags`."""
    h = ctypes.c_void_p()
    _check(load_library().asym_topology_load(path.encode(), key.encode(), flags, ctypes.byref(h)))
    return Topology(h.value)


def latency_params(**kw) -> LatencyParams:
    """Library defaults, with any field overridden by keyword."""
    p = LatencyParams()
    load_library().asym_latency_params_default(ctypes.byref(p))
    for k, v in kw.items():
        if not hasattr(p, k):
            raise TypeError(f"unknown latency parameter {k}")
        setattr(p, k, v)
    return p


def latency_probe(device: int = 0, want_raw: bool = False, **kw):
    """Run the per-XCD latency / affinity probe; returns the summary dict, and
    with want_raw the per-address minima as uint32 [3, n_xcds, n_samples]
    (regimes L2, memory-side cache, HBM)."""
    import numpy as np
    p = latency_params(**kw)
    s = LatencySummary()
    raw = None
    ptr = None
    if want_raw:
        n_x = device_query(device)["n_xccs"]
        raw = np.zeros((3, n_x, p.n_samples), dtype=np.uint32)
        ptr = raw.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))
    _check(load_library().asym_latency_probe(device, ctypes.byref(p), ptr, ctypes.byref(s)))
    d = s.to_dict()
    return (d, raw) if want_raw else d


def latency_analyze(hbm_lat, group_threshold: float = 0.5, tie_cycles: float = 20.0) -> dict:
    """Affinity analysis of uint32 [n_xcds, n_samples] HBM latencies (host only)."""
    import numpy as np
    L = np.ascontiguousarray(hbm_lat, dtype=np.uint32)
    if L.ndim != 2:
        raise ValueError("latencies must be [n_xcds, n_samples]")
    s = LatencySummary()
    _check(load_library().asym_latency_analyze(L.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)),
                                               L.shape[0], L.shape[1], group_threshold, tie_cycles,
                                               ctypes.byref(s)))
    return s.to_dict()


def interleave_params_default() -> dict:
    p = InterleaveParams()
    load_library().asym_interleave_params_default(ctypes.byref(p))
    return {k: getattr(p, k) for k, _ in p._fields_}


def interleave_probe(device: int = 0, **kw):
    """Run the partition-hash probe; returns (result dict, offsets uint64 [n],
    HBM latencies uint32 [n_xcds, n], homes int8 [n])."""
    import numpy as np
    p = InterleaveParams()
    load_library().asym_interleave_params_default(ctypes.byref(p))
    for k, v in kw.items():
        if not hasattr(p, k):
            raise TypeError(f"unknown interleave parameter {k}")
        setattr(p, k, v)
    n = p.n_bases * (1 + p.hi_bit - p.lo_bit + p.n_pairs)
    n_x = device_query(device)["n_xccs"]
    offs = np.zeros(n, dtype=np.uint64)
    lat = np.zeros((n_x, n), dtype=np.uint32)
    home = np.zeros(n, dtype=np.int8)
    r = InterleaveResult()
    _check(load_library().asym_interleave_probe(
        device, ctypes.byref(p), offs.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
        lat.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)),
        home.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)), ctypes.byref(r)))
    return r.to_dict(), offs, lat, home


def interleave_analyze(hbm_lat, offs, block: int, group_threshold: float = 0.5,
                       tie_cycles: float = 20.0, decide: float = 0.1) -> dict:
    """Partition-hash analysis of uint32 [n_xcds, n] HBM latencies over byte
    offsets [n] in blocks of `block` (host only); the dict carries the homes."""
    import numpy as np
    L = np.ascontiguousarray(hbm_lat, dtype=np.uint32)
    o = np.ascontiguousarray(offs, dtype=np.uint64)
    if L.ndim != 2 or o.ndim != 1:
        raise ValueError("latencies must be [n_xcds, n] and offsets [n]")
    if L.shape[1] != o.shape[0]:
        raise ValueError("latency columns and offsets differ in count")
    home = np.zeros(o.shape[0], dtype=np.int8)
    r = InterleaveResult()
    _check(load_library().asym_interleave_analyze(
        L.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), L.shape[0], o.shape[0],
        o.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), block, group_threshold, tie_cycles, decide,
        home.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)), ctypes.byref(r)))
    d = r.to_dict()
    d["home"] = [int(h) for h in home]
    return d


def home_map(ptr: int, nbytes: int, hash_mask: int, chunk_log2: int, group_of_xcd=None,
             passes: int = 4, n_verify: int = 1024, seed: int = 1, tie_cycles: float = 20.0,
             device: int = 0):
    """Home group of every 2^chunk_log2-byte chunk of the device range [ptr,
    ptr + nbytes) (both multiples of 2 MiB); returns (info dict, int8 homes)."""
    import numpy as np
    homes = np.zeros(nbytes >> chunk_log2, dtype=np.int8)
    info = HomeMapInfo()
    g = _ints(group_of_xcd) if group_of_xcd is not None else None
    _check(load_library().asym_home_map(device, ctypes.c_void_p(ptr), nbytes, hash_mask, chunk_log2, g,
                                        passes, n_verify, seed, tie_cycles,
                                        homes.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)),
                                        ctypes.byref(info)))
    n_x = len(group_of_xcd) if group_of_xcd is not None else device_query(device)["n_xccs"]
    return info.to_dict(n_x), homes


def home_map_analyze(lat, n_pages: int, verify_offs, group_of_xcd, hash_mask: int, chunk_log2: int,
                     tie_cycles: float = 20.0):
    """Host analysis of page-line and verification-line latencies [n_xcds,
    n_pages + n_verify]; returns (info dict, int8 homes)."""
    import numpy as np
    L = np.ascontiguousarray(lat, dtype=np.uint32)
    vo = np.ascontiguousarray(verify_offs, dtype=np.uint64)
    if L.ndim != 2 or L.shape[1] != n_pages + vo.shape[0]:
        raise ValueError("latencies must be [n_xcds, n_pages + n_verify]")
    homes = np.zeros((n_pages << 21) >> chunk_log2, dtype=np.int8)
    info = HomeMapInfo()
    _check(load_library().asym_home_map_analyze(
        L.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)), L.shape[0], n_pages,
        vo.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), vo.shape[0], _ints(group_of_xcd), hash_mask,
        chunk_log2, tie_cycles, homes.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)), ctypes.byref(info)))
    return info.to_dict(L.shape[0]), homes


def chunk_lists(homes, n_xcds: int, group_of_xcd, mode: int, xcd_mask: int = 0):
    """(chunk indices XCD by XCD as uint32, offsets [n_xcds + 1] as int32)."""
    import numpy as np
    h = np.ascontiguousarray(homes, dtype=np.int8)
    out = np.zeros(max(1, h.shape[0]), dtype=np.uint32)
    off = np.zeros(n_xcds + 1, dtype=np.int32)
    n = ctypes.c_int()
    g = _ints(group_of_xcd) if group_of_xcd is not None else None
    _check(load_library().asym_chunk_lists(
        h.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)), h.shape[0], n_xcds, g, xcd_mask, mode,
        out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32)),
        off.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), ctypes.byref(n)))
    return out[:n.value], off


def chunk_read_bw(ptr: int, nbytes: int, chunk_log2: int, chunks, off, iters: int = 5, stream=None,
                  workers_per_xcd: Optional[int] = None):
    """Read the listed chunks of [ptr, ptr + nbytes) `iters` times (256
    workgroups per XCD, or workers_per_xcd); returns (ms per iteration, XOR of
    every 16-byte word read as 4 uint32)."""
    import numpy as np
    c = np.ascontiguousarray(chunks, dtype=np.uint32)
    o = np.ascontiguousarray(off, dtype=np.int32)
    ms = ctypes.c_double()
    ck = np.zeros(4, dtype=np.uint32)
    cp_ = c.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))
    op_ = o.ctypes.data_as(ctypes.POINTER(ctypes.c_int))
    ckp = ck.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))
    if workers_per_xcd is None:
        _check(load_library().asym_chunk_read_bw(ctypes.c_void_p(ptr), nbytes, chunk_log2, cp_, op_, o.shape[0] - 1,
                                                 iters, _stream_ptr(stream), ckp, ctypes.byref(ms)))
    else:
        _check(load_library().asym_chunk_read(ctypes.c_void_p(ptr), nbytes, chunk_log2, cp_, op_, o.shape[0] - 1,
                                              workers_per_xcd, iters, _stream_ptr(stream), ckp, ctypes.byref(ms)))
    return ms.value, ck


def topology_from_records(records, n_cus: int, n_xccs: int, mask_bit_record=None) -> Topology:
    import numpy as np
    rec = np.ascontiguousarray(records, dtype=np.int32).reshape(-1, 4)
    mb = None
    if mask_bit_record is not None:
        mb = np.ascontiguousarray(mask_bit_record, dtype=np.int32)
    h = ctypes.c_void_p()
    _check(load_library().asym_topology_from_records(
        rec.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), rec.shape[0], n_cus, n_xccs,
        mb.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)) if mb is not None else None,
        ctypes.byref(h)))
    return Topology(h.value)


# ---- schedule ----------------------------------------------------------------

def schedule_build(tiles_m: int, tiles_n: int, slots: Sequence[int], mapping: int, band: int = 0):
    n_x = len(slots)
    T = tiles_m * tiles_n
    order = (ctypes.c_int * T)()
    off = (ctypes.c_int * (n_x + 1))()
    quota = (ctypes.c_int * n_x)()
    _check(load_library().asym_schedule_build(tiles_m, tiles_n, n_x, _ints(slots), mapping, band,
                                              order, off, quota))
    return list(order), list(off), list(quota)


def grouped_schedule_build(tiles_m: Sequence[int], tiles_n: int, slots: Sequence[int], mapping: int):
    n_x = len(slots)
    T = sum(tiles_m) * tiles_n
    order = (ctypes.c_int * max(1, T))()
    off = (ctypes.c_int * (n_x + 1))()
    quota = (ctypes.c_int * n_x)()
    _check(load_library().asym_grouped_schedule_build(len(tiles_m), _ints(tiles_m), tiles_n, n_x,
                                                      _ints(slots), mapping, order, off, quota))
    return list(order)[:T], list(off), list(quota)


# ---- streams ---------------------------------------------------------------------

def stream_create(topo: Optional[Topology] = None, mask: Optional[Sequence[int]] = None):
    """A library stream (optionally CU-masked) wrapped as torch.cuda.ExternalStream."""
    import torch
    h = ctypes.c_void_p()
    _check(load_library().asym_stream_create(topo.handle if topo else None, mask_words(mask),
                                             ctypes.byref(h)))
    return torch.cuda.ExternalStream(h.value)


def stream_destroy(stream) -> None:
    _check(load_library().asym_stream_destroy(ctypes.c_void_p(stream.cuda_stream)))


def _stream_ptr(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# ---- GEMM -----------------------------------------------------------------------

def gemm(A, B, C=None, mapping="aware", topo: Optional[Topology] = None, xcd_mask: int = 0,
         stream=None, b_layout: str = "nk"):
    """C = A . B for bf16 CUDA tensors: A [M,K]; B [N,K] when b_layout is "nk"
    (its [N][K] storage: C = A . B^T of the tensor), or [K,N] when "kn".

    Launches the HIP kernels asynchronously on `stream` (default: torch's
    current stream) and returns C.
    """
    import torch
    if A.dtype != torch.bfloat16 or B.dtype != torch.bfloat16:
        raise TypeError("A and B must be bfloat16")
    if b_layout not in ("nk", "kn"):
        raise ValueError("b_layout must be 'nk' or 'kn'")
    kn = b_layout == "kn"
    if A.dim() != 2 or B.dim() != 2 or A.shape[1] != B.shape[0 if kn else 1]:
        raise ValueError("A must be [M,K] and B [K,N]" if kn else "A must be [M,K] and B [N,K]")
    if not (A.is_cuda and B.is_cuda):
        raise ValueError("A and B must be on the GPU")
    if A.stride(1) != 1 or B.stride(1) != 1:
        raise ValueError("A and B must be row-major (unit stride in their last dimension)")
    M, K = A.shape
    N = B.shape[1] if kn else B.shape[0]
    if C is None:
        C = torch.empty((M, N), dtype=torch.bfloat16, device=A.device)
    if C.dtype != torch.bfloat16 or C.shape != (M, N) or C.stride(1) != 1:
        raise ValueError("C must be a row-major bf16 [M,N] tensor")
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    _check(load_library().asym_gemm_bf16(
        topo.handle if topo else None, M, N, K, ctypes.c_void_p(A.data_ptr()), A.stride(0),
        ctypes.c_void_p(B.data_ptr()), B.stride(0), B_KN if kn else B_NK, ctypes.c_void_p(C.data_ptr()),
        C.stride(0), mp, xcd_mask, _stream_ptr(stream)))
    return C


def gemm_noalloc(A, B, C, topo: "Topology", mapping="aware", xcd_mask: int = 0, stream=None):
    """gemm() through the entry point that allocates no device memory (its
    schedule, counters and split-K partials sit in the library's fixed
    per-GPU array): A [M,K], B [N,K], C [M,N] bf16 CUDA tensors, all given;
    topo must be a probed topology.  Calls that overlap on one GPU race."""
    import torch
    if A.dtype != torch.bfloat16 or B.dtype != torch.bfloat16 or C.dtype != torch.bfloat16:
        raise TypeError("A, B and C must be bfloat16")
    if A.dim() != 2 or B.dim() != 2 or A.shape[1] != B.shape[1]:
        raise ValueError("A must be [M,K] and B [N,K]")
    if A.stride(1) != 1 or B.stride(1) != 1 or C.stride(1) != 1:
        raise ValueError("A, B and C must be row-major")
    M, K = A.shape
    N = B.shape[0]
    if tuple(C.shape) != (M, N):
        raise ValueError("C must be [M,N]")
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    _check(load_library().asym_gemm_bf16_noalloc(
        topo.handle if topo else None, M, N, K, ctypes.c_void_p(A.data_ptr()), A.stride(0),
        ctypes.c_void_p(B.data_ptr()), B.stride(0), B_NK, ctypes.c_void_p(C.data_ptr()),
        C.stride(0), mp, xcd_mask, _stream_ptr(stream)))
    return C


def gemm_trace(A, B, C, mapping="aware", topo: Optional["Topology"] = None, xcd_mask: int = 0, stream=None,
               launches: int = 1):
    """gemm() on the persistent kernel with one record per workgroup (the
    48-byte asym_wg_record); returns a dict of numpy arrays indexed by block
    index: start, first_tile, end (constant-rate clock ticks), xcc, hw_id,
    tiles, worked, cycles (shader clock, start to end), and the launch plan.  With launches > 1 the launches are
    queued back to back, each with records of its own, and a list of such
    dicts comes back.  Synchronises the stream."""
    import numpy as np
    import torch
    M, K = A.shape
    N = B.shape[0]
    prev = set_small_m(False)  # the plan of the persistent kernel, which the trace runs
    try:
        plan = gemm_plan(A, B, C, mapping=mapping, topo=topo, xcd_mask=xcd_mask, stream=stream)
    finally:
        set_small_m(prev)
    grid = max(1, plan["grid"])
    rec = torch.zeros((launches, grid, 12), dtype=torch.int32, device=A.device)
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    lib = load_library()
    counts = []
    for i in range(launches):
        n = ctypes.c_int()
        _check(lib.asym_gemm_bf16_trace(
            topo.handle if topo else None, M, N, K, ctypes.c_void_p(A.data_ptr()), A.stride(0),
            ctypes.c_void_p(B.data_ptr()), B.stride(0), B_NK, ctypes.c_void_p(C.data_ptr()), C.stride(0), mp,
            xcd_mask, _stream_ptr(stream), ctypes.c_void_p(rec[i].data_ptr()), grid, ctypes.byref(n)))
        counts.append(n.value)
    (stream if stream is not None else torch.cuda.current_stream()).synchronize()
    host = rec.cpu().numpy().view(np.uint32)
    out = []
    for i in range(launches):
        r = host[i, : counts[i]]
        u64 = lambda lo: r[:, lo].astype(np.uint64) | (r[:, lo + 1].astype(np.uint64) << np.uint64(32))
        out.append({"start": u64(0), "first_tile": u64(2), "end": u64(4), "xcc": r[:, 6].copy(),
                    "hw_id": r[:, 7].copy(), "tiles": r[:, 8].copy(), "worked": r[:, 9].copy(),
                    "cycles": u64(10), "plan": plan})
    return out[0] if launches == 1 else out


def noalloc_limits() -> dict:
    """The per-GPU array of gemm_noalloc: its size, the most output tiles and
    the most split-K partial bytes a call may need."""
    sb, pb = ctypes.c_size_t(), ctypes.c_size_t()
    mt = ctypes.c_int()
    _check(load_library().asym_gemm_noalloc_limits(ctypes.byref(sb), ctypes.byref(mt), ctypes.byref(pb)))
    return {"scratch_bytes": sb.value, "max_tiles": mt.value, "max_partial_bytes": pb.value}


def gemm_grouped(A, B, M: Sequence[int], C=None, mapping="aware", topo: Optional[Topology] = None,
                 xcd_mask: int = 0, stream=None):
    """Grouped GEMM: C_g = A_g . B_g^T for every group g, one launch.

    A: bf16 CUDA tensor [sum(M), K], the groups' rows packed in group order.
    B: bf16 CUDA tensor [G, N, K] (or [G * N, K]), group g's weights [N, K].
    M: the G row counts.  Returns C [sum(M), N], packed like A.
    """
    import torch
    G = len(M)
    if A.dtype != torch.bfloat16 or B.dtype != torch.bfloat16:
        raise TypeError("A and B must be bfloat16")
    if not (A.is_cuda and B.is_cuda):
        raise ValueError("A and B must be on the GPU")
    if B.dim() == 3:
        if B.shape[0] != G:
            raise ValueError("B must be [G, N, K]")
        N, K = B.shape[1], B.shape[2]
        if not B.is_contiguous():
            raise ValueError("B [G, N, K] must be contiguous")
        ldb = K
    elif B.dim() == 2:
        if B.shape[0] % G:
            raise ValueError("B [G * N, K]: rows not a multiple of G")
        N, K = B.shape[0] // G, B.shape[1]
        if B.stride(1) != 1:
            raise ValueError("B must be K-contiguous")
        ldb = B.stride(0)
    else:
        raise ValueError("B must be [G, N, K] or [G * N, K]")
    rows = int(sum(M))
    if A.dim() != 2 or A.shape[0] != rows or A.shape[1] != K or A.stride(1) != 1:
        raise ValueError("A must be a K-contiguous [sum(M), K] tensor")
    if C is None:
        C = torch.empty((rows, N), dtype=torch.bfloat16, device=A.device)
    if C.dtype != torch.bfloat16 or tuple(C.shape) != (rows, N) or C.stride(1) != 1:
        raise ValueError("C must be a row-major bf16 [sum(M), N] tensor")
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    _check(load_library().asym_gemm_grouped_bf16(
        topo.handle if topo else None, G, _ints([int(m) for m in M]), N, K,
        ctypes.c_void_p(A.data_ptr()), max(A.stride(0), K), ctypes.c_void_p(B.data_ptr()), ldb,
        ctypes.c_void_p(C.data_ptr()), max(C.stride(0), N), mp, xcd_mask, _stream_ptr(stream)))
    return C


def attn_decode(q, k, v, o=None, lse=None, scale: Optional[float] = None, split_tokens: int = 0,
                mapping="aware", topo: Optional[Topology] = None, xcd_mask: int = 0, stream=None):
    """Decode attention: q [B, H_q, D], k and v [B, H_kv, S_k, D] bf16 CUDA
    tensors (contiguous); returns O [B, H_q, D] bf16 (and fills lse [B, H_q]
    fp32 when given).  scale defaults to 1 / sqrt(D)."""
    import math

    import torch
    if q.dtype != torch.bfloat16 or k.dtype != torch.bfloat16 or v.dtype != torch.bfloat16:
        raise TypeError("q, k, v must be bfloat16")
    if not (q.is_cuda and k.is_cuda and v.is_cuda):
        raise ValueError("q, k, v must be on the GPU")
    if q.dim() != 3 or k.dim() != 4 or v.shape != k.shape:
        raise ValueError("q must be [B, H_q, D] and k, v [B, H_kv, S_k, D]")
    if not (q.is_contiguous() and k.is_contiguous() and v.is_contiguous()):
        raise ValueError("q, k, v must be contiguous")
    B, Hq, D = q.shape
    Bk, Hkv, S, Dk = k.shape
    if Bk != B or Dk != D:
        raise ValueError("q and k disagree on B or D")
    if o is None:
        o = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=q.device)
    if o.dtype != torch.bfloat16 or tuple(o.shape) != (B, Hq, D) or not o.is_contiguous():
        raise ValueError("o must be a contiguous bf16 [B, H_q, D] tensor")
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, Hq) or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous fp32 [B, H_q] tensor")
    sc = 1.0 / math.sqrt(D) if scale is None else float(scale)
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    _check(load_library().asym_attn_decode_bf16(
        topo.handle if topo else None, B, Hq, Hkv, S, D, ctypes.c_void_p(q.data_ptr()),
        ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(o.data_ptr()),
        ctypes.c_void_p(lse.data_ptr() if lse is not None else None), sc, split_tokens, mp, xcd_mask,
        _stream_ptr(stream)))
    return o


PAGES_IN_ORDER, PAGES_LOCAL, PAGES_REMOTE = 0, 1, 2
PAGE_TOKENS = 32  # tokens of one head per 8 KiB page of the paged cache


def attn_decode_paged(q, k_pool, v_pool, k_pages, v_pages, S: int, o=None, lse=None, scale: Optional[float] = None,
                      split_tokens: int = 0, mapping="aware", topo: Optional[Topology] = None, xcd_mask: int = 0,
                      stream=None):
    """Decode attention over a paged cache: q [B, H_q, 128] bf16; k_pool and
    v_pool bf16 [pool_pages, 32, 128]; k_pages and v_pages int32 CUDA tensors
    [B, H_kv, ceil(S / 32)] naming each (request, head, page)'s pool page.
    Returns O [B, H_q, 128] bf16 (and fills lse when given), as attn_decode
    on the dense K and V the tables describe."""
    import math

    import torch
    if q.dtype != torch.bfloat16 or k_pool.dtype != torch.bfloat16 or v_pool.dtype != torch.bfloat16:
        raise TypeError("q and the pools must be bfloat16")
    if k_pages.dtype != torch.int32 or v_pages.dtype != torch.int32:
        raise TypeError("page tables must be int32")
    if not all(t.is_cuda and t.is_contiguous() for t in (q, k_pool, v_pool, k_pages, v_pages)):
        raise ValueError("q, the pools and the tables must be contiguous GPU tensors")
    if q.dim() != 3 or q.shape[2] != 128:
        raise ValueError("q must be [B, H_q, 128]")
    if k_pool.shape != v_pool.shape or k_pool.dim() != 3 or tuple(k_pool.shape[1:]) != (PAGE_TOKENS, 128):
        raise ValueError("pools must be [pool_pages, 32, 128]")
    B, Hq, _ = q.shape
    if k_pages.dim() != 3 or k_pages.shape != v_pages.shape or k_pages.shape[0] != B \
            or k_pages.shape[2] != (S + PAGE_TOKENS - 1) // PAGE_TOKENS:
        raise ValueError("page tables must be [B, H_kv, ceil(S / 32)]")
    Hkv = k_pages.shape[1]
    if o is None:
        o = torch.empty((B, Hq, 128), dtype=torch.bfloat16, device=q.device)
    if o.dtype != torch.bfloat16 or tuple(o.shape) != (B, Hq, 128) or not o.is_contiguous():
        raise ValueError("o must be a contiguous bf16 [B, H_q, 128] tensor")
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, Hq) or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous fp32 [B, H_q] tensor")
    sc = 1.0 / math.sqrt(128) if scale is None else float(scale)
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    _check(load_library().asym_attn_decode_paged_bf16(
        topo.handle if topo else None, B, Hq, Hkv, S, ctypes.c_void_p(q.data_ptr()),
        ctypes.c_void_p(k_pool.data_ptr()), ctypes.c_void_p(v_pool.data_ptr()), k_pool.shape[0],
        ctypes.c_void_p(k_pages.data_ptr()), ctypes.c_void_p(v_pages.data_ptr()), ctypes.c_void_p(o.data_ptr()),
        ctypes.c_void_p(lse.data_ptr() if lse is not None else None), sc, split_tokens, mp, xcd_mask,
        _stream_ptr(stream)))
    return o


def attn_pages_place(plan: dict, B: int, Hkv: int, S: int, pool_pages: int, policy: int = PAGES_IN_ORDER,
                     pool_home=None, group_of_xcd=None):
    """Page table (numpy int32 [B, H_kv, ceil(S / 32)]) for attn_decode_paged
    from an aware plan (attn_decode_plan) and the pool's page homes."""
    import numpy as np
    info = AttnPlanInfo()
    for k, _ in AttnPlanInfo._fields_:
        if k == "tasks_per_xcd":
            for x, v in enumerate(plan["tasks_per_xcd"]):
                info.tasks_per_xcd[x] = v
        else:
            setattr(info, k, plan.get(k, 0) if k == "dense_static" else plan[k])
    pph = (S + PAGE_TOKENS - 1) // PAGE_TOKENS
    out = np.zeros((B, Hkv, pph), dtype=np.int32)
    home = None
    if pool_home is not None:
        home = np.ascontiguousarray(pool_home, dtype=np.int8)
        if home.size < pool_pages:
            raise ValueError("pool_home must have pool_pages entries")
    grp = None
    if group_of_xcd is not None:
        grp = (ctypes.c_int * len(group_of_xcd))(*group_of_xcd)
    _check(load_library().asym_attn_pages_place(
        ctypes.byref(info), B, Hkv, S, home.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)) if home is not None else None,
        pool_pages, grp, policy, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
    return out


def attn_decode_plan(B: int, Hq: int, Hkv: int, S: int, D: int = 128, split_tokens: int = 0,
                     mapping="aware", topo: Optional[Topology] = None, xcd_mask: int = 0, stream=None) -> dict:
    out = AttnPlanInfo()
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    _check(load_library().asym_attn_decode_plan(topo.handle if topo else None, B, Hq, Hkv, S, D, split_tokens,
                                                mp, xcd_mask, _stream_ptr(stream), ctypes.byref(out)))
    return out.to_dict()


def set_mla_workgroup_form(level) -> int:
    """Which kernel forms mla_decode may take, for the process: 0 (or False)
    the wave form only, 1 up to the 64-head workgroup form, 2 (or True, the
    default) also the 128-head form where it has enough tasks, 3 the 128-head
    form wherever the head count allows; returns the previous level."""
    lvl = 2 if level is True else 0 if level is False else int(level)
    prev = load_library().asym_mla_set_workgroup_form(lvl)
    if prev < 0:
        _check(prev)
    return prev


def set_small_m(enable: bool) -> bool:
    """Switch the small-M kernel on or off for the process; returns the previous setting."""
    return bool(load_library().asym_gemm_set_small_m(1 if enable else 0))


def gemm_plan(A=None, B=None, C=None, mapping="aware", topo: Optional[Topology] = None,
              xcd_mask: int = 0, stream=None, M: Optional[int] = None, N: Optional[int] = None,
              K: Optional[int] = None, b_layout: str = "nk") -> dict:
    """What gemm() would launch for these operands (or, given M, N, K alone,
    for dense 256-byte-aligned operands of that shape): tile shape and grid,
    workers in all and per XCD, static or claiming aware form, vector or
    predicated path.  Launches nothing."""
    kn = b_layout == "kn"
    if A is not None:
        M, K = A.shape
        N = B.shape[1] if kn else B.shape[0]
        pa, lda = A.data_ptr(), A.stride(0)
        pb, ldb = B.data_ptr(), B.stride(0)
        if C is not None:
            pc, ldc = C.data_ptr(), C.stride(0)
        else:
            pc, ldc = 256, N
    else:
        if M is None or N is None or K is None:
            raise ValueError("give A and B, or M, N and K")
        pa, lda, pb, ldb, pc, ldc = 256, K, 256, (N if kn else K), 256, N
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    out = GemmPlanInfo()
    _check(load_library().asym_gemm_plan(
        topo.handle if topo else None, M, N, K, ctypes.c_void_p(pa), lda, ctypes.c_void_p(pb),
        ldb, B_KN if kn else B_NK, ctypes.c_void_p(pc), ldc, mp, xcd_mask, _stream_ptr(stream),
        ctypes.byref(out)))
    return out.to_dict()


def mla_decode(q, kv, o=None, lse=None, scale: Optional[float] = None, split_tokens: int = 0,
               mapping="aware", topo: Optional[Topology] = None, xcd_mask: int = 0, stream=None):
    """Latent-attention decode: q [B, H_q, 576] and the cache kv [B, S_k, 576]
    bf16 CUDA tensors (contiguous); returns O [B, H_q, 512] bf16 (and fills
    lse [B, H_q] fp32 when given).  scale defaults to 1 / sqrt(192)."""
    import math
    import torch
    if q.dtype != torch.bfloat16 or kv.dtype != torch.bfloat16:
        raise TypeError("q and kv must be bfloat16")
    if q.dim() != 3 or kv.dim() != 3 or q.shape[2] != 576 or kv.shape[2] != 576 or q.shape[0] != kv.shape[0]:
        raise ValueError("q must be [B, H_q, 576] and kv [B, S_k, 576]")
    if not (q.is_contiguous() and kv.is_contiguous()):
        raise ValueError("q and kv must be contiguous")
    B, Hq, _ = q.shape
    S = kv.shape[1]
    if o is None:
        o = torch.empty((B, Hq, 512), dtype=torch.bfloat16, device=q.device)
    if o.dtype != torch.bfloat16 or tuple(o.shape) != (B, Hq, 512) or not o.is_contiguous():
        raise ValueError("o must be a contiguous bf16 [B, H_q, 512] tensor")
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, Hq) or not lse.is_contiguous()):
        raise ValueError("lse must be a contiguous fp32 [B, H_q] tensor")
    sc = 1.0 / math.sqrt(192.0) if scale is None else float(scale)
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    _check(load_library().asym_mla_decode_bf16(
        topo.handle if topo else None, B, Hq, S, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(kv.data_ptr()),
        ctypes.c_void_p(o.data_ptr()), ctypes.c_void_p(lse.data_ptr()) if lse is not None else None, sc,
        split_tokens, mp, xcd_mask, _stream_ptr(stream)))
    return o


def mla_decode_plan(B: int, Hq: int, S: int, split_tokens: int = 0, mapping="aware",
                    topo: Optional[Topology] = None, xcd_mask: int = 0, stream=None) -> dict:
    mp = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    out = MlaPlanInfo()
    _check(load_library().asym_mla_decode_plan(topo.handle if topo else None, B, Hq, S, split_tokens, mp,
                                               xcd_mask, _stream_ptr(stream), ctypes.byref(out)))
    return out.to_dict()


# ---- copy and co-run --------------------------------------------------------------

def copy(dst, src, passes: int = 1, stop_flag=None, xcd_mask: int = 0, stream=None,
         topo: Optional["Topology"] = None):
    """`passes` streaming copies of the CUDA tensor src into dst (same byte
    size) on `stream`'s CU set; stop_flag: an int32 CUDA tensor or None."""
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != n:
        raise ValueError("size mismatch")
    _check(load_library().asym_copy_bf16(
        topo.handle if topo else None,
        ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()), n, passes,
        ctypes.c_void_p(stop_flag.data_ptr()) if stop_flag is not None else None, xcd_mask,
        _stream_ptr(stream)))
    return dst


def gemm_task(A, B, C, iters: int, mapping="aware", mask=None, xcd_mask: int = 0, warm_iters: int = 0) -> Task:
    t = Task()
    t.warm_iters = warm_iters
    t.kind = 0
    if mask is not None:
        m = mask_words(mask)
        for w in range(MASK_WORDS):
            t.mask[w] = m[w]
    t.xcd_mask = xcd_mask
    t.iters = iters
    t.mapping = MAPPINGS[mapping] if isinstance(mapping, str) else int(mapping)
    t.M, t.K = A.shape
    t.N = B.shape[0]
    t.A, t.B, t.C = A.data_ptr(), B.data_ptr(), C.data_ptr()
    return t


def copy_task(dst, src, passes: int, mask=None, xcd_mask: int = 0, grid: int = 0, warm_passes: int = 0) -> Task:
    """The streaming-copy tenant: `passes` copies of src into dst (after
    `warm_passes` untimed ones)."""
    t = Task()
    t.warm_iters = warm_passes
    t.kind = 1
    t.grid = grid
    if mask is not None:
        m = mask_words(mask)
        for w in range(MASK_WORDS):
            t.mask[w] = m[w]
    t.xcd_mask = xcd_mask
    t.iters = passes
    t.src, t.dst = src.data_ptr(), dst.data_ptr()
    t.n_bytes = src.numel() * src.element_size()
    return t


def read_task(src, passes: int, mask=None, xcd_mask: int = 0, grid: int = 0, warm_passes: int = 0) -> Task:
    """A bandwidth-bound co-runner: `passes` whole reads of the CUDA tensor src,
    on `grid` workgroups (0: 8 per CU of its XCD with the most CUs, on every XCD),
    after `warm_passes` untimed ones."""
    t = Task()
    t.warm_iters = warm_passes
    t.grid = grid
    t.kind = 2
    if mask is not None:
        m = mask_words(mask)
        for w in range(MASK_WORDS):
            t.mask[w] = m[w]
    t.xcd_mask = xcd_mask
    t.iters = passes
    t.src = src.data_ptr()
    t.n_bytes = src.numel() * src.element_size()
    return t


def corun(tasks: Sequence[Task], topo: Optional[Topology] = None) -> list:
    n = len(tasks)
    arr = (Task * n)(*tasks)
    res = (TaskResult * n)()
    _check(load_library().asym_corun(topo.handle if topo else None, arr, n, res))
    out = [{k: getattr(r, k) for k, _ in TaskResult._fields_} for r in res]
    for d in out:
        d["checksum"] = list(d["checksum"])
    return out


def last_error() -> str:
    return load_library().asym_last_error().decode()


def version() -> int:
    return load_library().asym_version()
