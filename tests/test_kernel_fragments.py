"""In-flight fragment registers in the compiled GEMM (CPU only: hipcc -S for gfx950).

The ring's MFMA fragments are read from LDS by inline-asm ds_read_b128: the
compiler does not know that the destination registers are written later, when
the read completes, and the kernel's own `s_waitcnt lgkmcnt(0)` is the wait.
If the compiler copies, reads or reuses such a register before that wait
(for instance to reconcile register assignments where two paths join), the
copy takes the stale value and the product is wrong; this went wrong once
when a loop body got two paths.  The test runs a dataflow pass over the
control-flow graph of each vector-path kernel and requires that no
instruction touches a fragment register between the read that fills it and
the next lgkmcnt(0).  The accumulators have the same problem with the
inline-asm MFMAs that write them: reading them needs the wait states of the
kernel's MFMA fence (`s_nop 7` x 3), which the compiler does not know about, so
no instruction the compiler places may touch an accumulator register between
an MFMA and the fence.  The other direction, an accumulator the compiler writes
(zeroing, a rescale) and an inline-asm MFMA that then reads it, needs a few
wait states too: every path from such a write to such an MFMA must carry at
least `MIN_WRITE_TO_MFMA` of them.  Both checks also run over the latent-
attention decode kernel whose 128-head form keeps its outputs in AGPRs
through inline-asm MFMAs.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_24270_amd", "csrc")

_VREG = re.compile(r"\bv(?:\[(\d+):(\d+)\]|(\d+)\b)")
# instructions whose first operand is read, not written
_NO_DEST = re.compile(r"^(buffer_store|global_store|flat_store|scratch_store|ds_write|ds_store|"
                      r"buffer_load\w*.*\blds\b|s_\w+|v_cmpx)")


def _vregs(text: str):
    out = set()
    for m in _VREG.finditer(text):
        if m.group(3) is not None:
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def _split(inst: str):
    """(mnemonic, written VGPRs, read VGPRs) of one instruction."""
    inst = inst.split(";")[0].strip()
    parts = inst.split(None, 1)
    mn = parts[0]
    ops = parts[1] if len(parts) > 1 else ""
    args = [a.strip() for a in ops.split(",")]
    if _NO_DEST.match(inst) or not args or not args[0]:
        return mn, set(), _vregs(ops)
    dst, srcs = args[0], ",".join(args[1:])
    reads = _vregs(srcs)
    writes = _vregs(dst)
    if mn.startswith(("v_permlane16_swap", "v_permlane32_swap", "v_writelane")):
        reads |= writes  # swaps and lane writes also read their first operand
    return mn, writes, reads


def blocks_of(asm: str, kernel: str):
    lines = asm.splitlines()
    start = next(i for i, l in enumerate(lines) if re.match(r"^" + re.escape(kernel) + r":", l))
    end = next(i for i in range(start, len(lines)) if lines[i].startswith(".Lfunc_end"))
    blocks, cur, in_asm = [], {"label": None, "insts": []}, False
    for l in lines[start + 1:end]:
        st = l.strip()
        m = re.match(r"^(\.LBB\d+_\d+):", st)
        if m or re.match(r"^; %bb\.\d+:", st):
            if cur["insts"] or cur["label"]:
                blocks.append(cur)
            cur = {"label": m.group(1) if m else None, "insts": []}
            continue
        if st.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if st.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if not st or st.startswith(";") or st.startswith("."):
            continue
        for piece in st.split("\n"):
            cur["insts"].append((piece.strip(), in_asm))
    blocks.append(cur)
    return blocks


def successors(blocks):
    label_at = {b["label"]: i for i, b in enumerate(blocks) if b["label"]}
    succ = []
    for i, b in enumerate(blocks):
        last = b["insts"][-1][0] if b["insts"] else ""
        m = re.match(r"^s_(c?branch\w*)\s+(\.LBB\d+_\d+)", last)
        s = []
        if last.startswith("s_endpgm"):
            pass
        elif m and m.group(1) == "branch":
            s = [label_at[m.group(2)]]
        elif m:
            s = [label_at[m.group(2)]] + ([i + 1] if i + 1 < len(blocks) else [])
        elif i + 1 < len(blocks):
            s = [i + 1]
        succ.append(s)
    return succ


_AGPR_TOUCH = re.compile(r"^v_accvgpr_(read|write|mov)")


def transfer(block, state, violations=None):
    """state: (VGPRs whose fragment read is in flight, MFMA results pending)."""
    cur, mfma = set(state[0]), state[1]
    nops = 0
    for inst, is_asm in block["insts"]:
        mn, writes, reads = _split(inst)
        if is_asm and mn == "s_nop" and inst.split()[-1] == "7":
            nops += 1
            if nops >= 3:
                mfma = False
            continue
        nops = 0
        if mn == "s_waitcnt":
            m = re.search(r"lgkmcnt\((\d+)\)", inst)
            if m and int(m.group(1)) == 0:
                cur.clear()
            continue
        if is_asm and mn == "ds_read_b128":
            cur |= writes
            continue
        if is_asm and mn.startswith("v_mfma"):
            mfma = True
        elif mfma and not is_asm and _AGPR_TOUCH.match(mn) and violations is not None:
            violations.append((block["label"], inst, "accumulator touched before the MFMA fence"))
        bad = (reads | writes) & cur
        if bad and violations is not None:
            violations.append((block["label"], inst, sorted(bad)))
    return cur, mfma


def inflight_violations(asm: str, kernel: str):
    blocks = blocks_of(asm, kernel)
    succ = successors(blocks)
    ins = [(set(), False) for _ in blocks]
    changed = True
    while changed:
        changed = False
        for i, b in enumerate(blocks):
            out = transfer(b, ins[i])
            for j in succ[i]:
                merged = (ins[j][0] | out[0], ins[j][1] or out[1])
                if merged != ins[j]:
                    ins[j] = merged
                    changed = True
    v = []
    for i, b in enumerate(blocks):
        transfer(b, ins[i], v)
    return v


def _compile(tmp_path_factory, src):
    out = tmp_path_factory.mktemp("asm") / (src + ".s")
    cmd = ["hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-I", os.path.join(ROOT, "include"),
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-mllvm", "-amdgpu-mfma-vgpr-form=1",
           "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return out.read_text()


@pytest.fixture(scope="module")
def gemm_asm(tmp_path_factory):
    return _compile(tmp_path_factory, "gemm.hip")


@pytest.fixture(scope="module")
def mla_asm(tmp_path_factory):
    return _compile(tmp_path_factory, "mla_decode.hip")


MLA_128 = "_ZN4asym12_GLOBAL__N_119mla_decode_split_wgILi2EEEvNS0_9MlaParamsE"
MIN_WRITE_TO_MFMA = 4


def write_to_mfma_violations(asm: str, kernel: str):
    """Inline-asm MFMAs reached from a compiler-placed v_accvgpr_write by a
    path of fewer than MIN_WRITE_TO_MFMA wait states (s_nop n counts n + 1,
    any other instruction 1).  Dataflow over the control-flow graph: the
    state is the fewest wait states since such a write on any path."""
    blocks = blocks_of(asm, kernel)
    succ = successors(blocks)
    inf = 10 ** 9

    def tr(block, ws, out=None):
        for inst, is_asm in block["insts"]:
            mn = inst.split()[0]
            if is_asm and mn.startswith("v_mfma"):
                if ws < MIN_WRITE_TO_MFMA and out is not None:
                    out.append((block["label"], inst, ws))
                ws = min(inf, ws + 1)
            elif not is_asm and mn == "v_accvgpr_write_b32":
                ws = 0
            elif mn == "s_nop":
                ws = min(inf, ws + int(inst.split()[1]) + 1)
            else:
                ws = min(inf, ws + 1)
        return ws

    ins = [inf] * len(blocks)
    changed = True
    while changed:
        changed = False
        for i, b in enumerate(blocks):
            o = tr(b, ins[i])
            for j in succ[i]:
                if o < ins[j]:
                    ins[j] = o
                    changed = True
    v = []
    for i, b in enumerate(blocks):
        tr(b, ins[i], v)
    return v


@pytest.mark.parametrize("trace", [0, 1])
@pytest.mark.parametrize("nbf", [8, 7, 6])
def test_no_use_of_fragments_in_flight(gemm_asm, nbf, trace):
    kernel = f"_ZN4asym12_GLOBAL__N_120gemm_bf16_persistentILb1ELi{nbf}ELi0ELb{trace}EEEvNS0_6ParamsE"
    v = inflight_violations(gemm_asm, kernel)
    assert not v, f"{len(v)} instructions touch fragment registers still being read, e.g. {v[:4]}"


def test_mla_outputs_fenced(mla_asm):
    """The 128-head latent-attention kernel: no compiler-placed access of an
    output accumulator between an asm MFMA and the fence."""
    v = inflight_violations(mla_asm, MLA_128)
    assert not v, f"{len(v)} accumulator accesses before the MFMA fence, e.g. {v[:4]}"


@pytest.mark.parametrize("which", ["gemm8", "gemm7", "gemm6", "gemm8_trace", "mla128"])
def test_accumulator_writes_reach_asm_mfmas_late_enough(gemm_asm, mla_asm, which):
    if which == "mla128":
        asm, kernel = mla_asm, MLA_128
    else:
        nbf, trace = int(which[4]), int(which.endswith("trace"))
        asm, kernel = gemm_asm, f"_ZN4asym12_GLOBAL__N_120gemm_bf16_persistentILb1ELi{nbf}ELi0ELb{trace}EEEvNS0_6ParamsE"
    v = write_to_mfma_violations(asm, kernel)
    assert not v, f"{len(v)} asm MFMAs too soon after an accumulator write, e.g. {v[:3]}"


def test_write_to_mfma_rule_sees_a_short_path():
    """A write two instructions before an asm MFMA on one branch is flagged;
    with a fence in between it is not."""
    bad = """k:
\tv_accvgpr_write_b32 a0, 0
\ts_cbranch_scc1 .LBB0_2
.LBB0_1:
\ts_nop 7
.LBB0_2:
\t;;#ASMSTART
\tv_mfma_f32_16x16x32_bf16 a[0:3], v[0:3], v[4:7], a[0:3]
\t;;#ASMEND
\ts_endpgm
.Lfunc_end0:
"""
    v = write_to_mfma_violations(bad, "k")
    assert len(v) == 1 and v[0][2] == 1
    good = bad.replace("\ts_cbranch_scc1 .LBB0_2\n", "\ts_nop 7\n\ts_cbranch_scc1 .LBB0_2\n")
    assert write_to_mfma_violations(good, "k") == []


def test_checker_sees_a_planted_copy():
    """The pass flags a copy of a register whose read is in flight, across a
    branch, and accepts the same code with the wait in between."""
    bad = """k:
\t;;#ASMSTART
\tds_read_b128 v[10:13], v1 offset:0
\t;;#ASMEND
\ts_cbranch_scc1 .LBB0_2
.LBB0_1:
\tv_mov_b64_e32 v[20:21], v[12:13]
.LBB0_2:
\t;;#ASMSTART
\ts_waitcnt lgkmcnt(0)
\t;;#ASMEND
\ts_endpgm
.Lfunc_end0:
"""
    v = inflight_violations(bad, "k")
    assert len(v) == 1 and v[0][2] == [12, 13]
    # an accumulator read between an MFMA and the fence is flagged; after it, not
    mf = """k:
\t;;#ASMSTART
\tv_mfma_f32_16x16x32_bf16 a[0:3], v[0:3], v[4:7], a[0:3]
\t;;#ASMEND
\tv_accvgpr_read_b32 v9, a1
\t;;#ASMSTART
\ts_nop 7
\ts_nop 7
\ts_nop 7
\t;;#ASMEND
\tv_accvgpr_read_b32 v8, a0
\ts_endpgm
.Lfunc_end0:
"""
    v = inflight_violations(mf, "k")
    assert len(v) == 1 and "v9" in v[0][1]
    good = bad.replace("\ts_cbranch_scc1 .LBB0_2\n", "\ts_waitcnt lgkmcnt(0)\n\ts_cbranch_scc1 .LBB0_2\n")
    assert inflight_violations(good, "k") == []


# Scalar ALU instructions that write SCC (the add/sub/logic/shift/compare
# families); an inline asm that contains one must declare SCC clobbered, or
# the compiler may keep a live compare result in SCC across it.  (A missing
# clobber once turned a uniform select after a load into a select on the
# load's carry: the wrong B slot, wrong products.)
_SCC_WRITERS = re.compile(r"\bs_(add|addc|sub|subb|and|or|xor|andn2|orn2|nand|nor|xnor|lshl|lshr|ashr|bfe|"
                          r"min|max|cmp|bitcmp|abs|not)\w*\b")


def _asm_statements(src: str):
    """(template text, clobber text) of each `asm volatile(...)` / `asm(...)`."""
    out = []
    for m in re.finditer(r"\basm\s+(?:volatile\s*)?\(", src):
        i, depth = m.end(), 1
        while depth:
            depth += {"(": 1, ")": -1}.get(src[i], 0)
            i += 1
        body = src[m.end():i - 1]
        parts = re.split(r"(?<!:):(?!:)", body)
        template = "".join(re.findall(r'"((?:[^"\\]|\\.)*)"', parts[0]))
        clobbers = parts[3] if len(parts) > 3 else ""
        out.append((template, clobbers))
    return out


@pytest.mark.parametrize("src", sorted(f for f in os.listdir(CSRC) if f.endswith(".hip")))
def test_asm_that_writes_scc_declares_it(src):
    text = open(os.path.join(CSRC, src)).read()
    bad = [t for t, clob in _asm_statements(text) if _SCC_WRITERS.search(t) and '"scc"' not in clob]
    assert not bad, f"{src}: asm writing SCC without an scc clobber: {bad}"


def test_scc_rule_sees_a_missing_clobber():
    src = 'asm volatile("s_add_u32 %0, %1, %2" : "=s"(x) : "s"(a), "s"(b) : "memory");\n' \
          'asm volatile("s_add_u32 %0, %1, %2" : "=s"(x) : "s"(a), "s"(b) : "memory", "scc");\n' \
          'asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");\n'
    st = _asm_statements(src)
    flagged = [t for t, c in st if _SCC_WRITERS.search(t) and '"scc"' not in c]
    assert len(st) == 3 and len(flagged) == 1
