"""The ctypes mirrors of the C ABI's structs have the C layout (CPU only).

A small C program built with gcc against include/asym.h prints sizeof and the
offset of every field the Python side declares; both must match ctypes'.  The
per-workgroup trace record has no mirror (the binding reads it as 32-bit
words), so its size and offsets are checked against the word indices the
binding uses.
"""
import ctypes
import os
import subprocess

import pytest

import paper_2609_24270_amd as asym

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MIRRORS = {
    "asym_device_info": asym.DeviceInfo,
    "asym_latency_params": asym.LatencyParams,
    "asym_latency_summary": asym.LatencySummary,
    "asym_interleave_params": asym.InterleaveParams,
    "asym_interleave_result": asym.InterleaveResult,
    "asym_home_map_info": asym.HomeMapInfo,
    "asym_task": asym.Task,
    "asym_task_result": asym.TaskResult,
    "asym_gemm_plan_info": asym.GemmPlanInfo,
    "asym_attn_plan_info": asym.AttnPlanInfo,
    "asym_mla_plan_info": asym.MlaPlanInfo,
}

# the trace record's fields and the 32-bit word each starts at in the binding
TRACE_WORDS = {"start": 0, "first_tile": 2, "end": 4, "xcc": 6, "hw_id": 7, "tiles": 8, "worked": 9, "cycles": 10}


@pytest.fixture(scope="module")
def c_layout(tmp_path_factory):
    d = tmp_path_factory.mktemp("abi")
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "asym.h"', "int main(void) {"]
    items = [(c, [f for f, _ in py._fields_]) for c, py in MIRRORS.items()]
    items.append(("asym_wg_record", list(TRACE_WORDS)))
    for c, fields in items:
        lines.append(f'  printf("{c} size %zu\\n", sizeof({c}));')
        for f in fields:
            lines.append(f'  printf("{c} {f} %zu\\n", offsetof({c}, {f}));')
    lines += ["  return 0;", "}"]
    src = d / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = d / "layout"
    r = subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout
    layout = {}
    for ln in out.splitlines():
        name, field, val = ln.split()
        layout[(name, field)] = int(val)
    return layout


@pytest.mark.parametrize("cname", sorted(MIRRORS))
def test_mirror_matches_c(c_layout, cname):
    py = MIRRORS[cname]
    assert ctypes.sizeof(py) == c_layout[(cname, "size")], cname
    for f, _ in py._fields_:
        assert getattr(py, f).offset == c_layout[(cname, f)], (cname, f)


def test_trace_record_words(c_layout):
    assert c_layout[("asym_wg_record", "size")] == 48
    for f, w in TRACE_WORDS.items():
        assert c_layout[("asym_wg_record", f)] == 4 * w, f
