"""Structure of the compiled claim loops (CPU only: hipcc -S for gfx950).

The persistent GEMM claims work in a loop whose body holds barriers: one
lane claims, a barrier publishes the claim, every lane reads it.  If lane-
divergent code sits at the end of such a body, the compiler may restructure
the loop so that the barriers head an inner loop the claiming lane never
re-enters; the other lanes then keep re-reading a stale claim and the kernel
never ends.  These tests check, on the generated assembly, that each claim
atomic and the barrier that publishes it belong to the same loop.  The
streaming copy has no claims at all: no atomics, no barriers, no LDS.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_24270_amd", "csrc")


def asm_of(src: str, tmp_path) -> str:
    out = tmp_path / (os.path.basename(src) + ".s")
    cmd = ["hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-I", os.path.join(ROOT, "include"),
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           *(["-mllvm", "-amdgpu-mfma-vgpr-form=1"] if src == "gemm.hip" else []),
           "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return out.read_text()


def function_body(asm: str, name_fragment: str) -> list:
    lines = asm.splitlines()
    start = next(i for i, l in enumerate(lines)
                 if re.match(r"^_Z\w*" + name_fragment + r"\w*:", l))
    end = next(i for i in range(start, len(lines)) if lines[i].startswith(".Lfunc_end"))
    return lines[start:end]


def annotate_loops(body: list):
    """(instruction, innermost loop header, chain of enclosing headers) per
    instruction, from the loop comments the compiler writes on each block."""
    parent = {}
    out = []
    cur_loop, header_lbl, pending_parent = None, None, None
    for l in body:
        m = re.match(r"^(\.LBB\d+_\d+|; %bb\.\d+):", l)
        if m:
            header_lbl = m.group(1)[1:] if m.group(1).startswith(".") else None
            cur_loop = None
            mp = re.search(r"Parent Loop (BB\d+_\d+) Depth=", l)
            pending_parent = "L" + mp.group(1) if mp else None
            if re.search(r"Loop Header: Depth=", l):
                cur_loop = header_lbl
                if pending_parent:
                    parent.setdefault(header_lbl, pending_parent)
            mi = re.search(r"in Loop: Header=(BB\d+_\d+)", l)
            if mi:
                cur_loop = "L" + mi.group(1)
            continue
        st = l.strip()
        if st.startswith(";"):
            if re.search(r"Loop Header: Depth=", st) and header_lbl:
                cur_loop = header_lbl
                if pending_parent:
                    parent.setdefault(header_lbl, pending_parent)
            mp = re.search(r"Parent Loop (BB\d+_\d+) Depth=", st)
            if mp and header_lbl and cur_loop == header_lbl:
                parent.setdefault(header_lbl, "L" + mp.group(1))
            mi = re.search(r"in Loop: Header=(BB\d+_\d+)", st)
            if mi:
                cur_loop = "L" + mi.group(1)
            continue
        if st:
            out.append((st, cur_loop))

    def chain(h):
        c = []
        while h is not None:
            c.append(h)
            h = parent.get(h)
        return c
    return [(i, h, chain(h)) for (i, h) in out]


@pytest.fixture(scope="module")
def tmp(tmp_path_factory):
    return tmp_path_factory.mktemp("asm")


def test_copy_kernel_shares_nothing_between_workgroups(tmp):
    """The copy's work is fixed before launch: no atomic, no barrier, no LDS
    access and no scalar-cache write in the compiled kernel, so no wave waits
    on another and each ends after its bounded loops."""
    body = function_body(asm_of("copy.hip", tmp), "copy_kernel")
    text = "\n".join(body)
    insts = [i for (i, h, c) in annotate_loops(body)]
    assert any(i.startswith("global_load_dwordx4") for i in insts)
    assert any(i.startswith("global_store_dwordx4") for i in insts)
    assert not any("atomic" in i for i in insts), [i for i in insts if "atomic" in i]
    assert not any(i.startswith("s_barrier") for i in insts)
    assert not any(i.startswith("ds_") for i in insts)
    assert not re.search(r"\bs_(store|atomic|buffer_store|dcache_wb|scratch_store)", text)


def claims_published_in_their_loop(insts, claim_re):
    """For every claim atomic: if a loop enclosing it contains barriers, the
    outermost such loop must hold a barrier directly, not only inside a nested
    loop that the claim is not part of (the shape that never finishes)."""
    bar_chains = [c for (i, h, c) in insts if i.startswith("s_barrier")]
    bar_inner = {h for (i, h, c) in insts if i.startswith("s_barrier")}
    claims = [k for k, (i, h, c) in enumerate(insts) if re.match(claim_re, i)]
    assert claims
    checked = 0
    for k in claims:
        chain = insts[k][2]
        with_bars = [L for L in chain if any(L in bc for bc in bar_chains)]
        if not with_bars:
            continue            # a lane-local loop with no barrier anywhere in it
        outer = with_bars[-1]   # chains list loops innermost first
        assert outer in bar_inner, (k, chain, outer)
        checked += 1
    return checked


def test_gemm_tile_claim_is_published_in_its_own_loop(tmp):
    """The dynamic aware form claims tiles on per-XCD counters (offset 64 and
    up) inside the tile loop; every such claim must sit in the loop whose
    barrier publishes it.  No scalar-cache writes of any kind."""
    body = function_body(asm_of("gemm.hip", tmp), "gemm_bf16_persistentILb1ELi8ELi0ELb0E")
    insts = annotate_loops(body)
    n = claims_published_in_their_loop(insts, r"^global_atomic_add v\d+, v\d+, v\d+, s\[\d+:\d+\]( offset:\d+)? sc0")
    assert n >= 1
    text = "\n".join(body)
    assert not re.search(r"\bs_(store|atomic|buffer_store|dcache_wb|scratch_store)", text)
