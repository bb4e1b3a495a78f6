"""The decode kernels issue some global loads with inline asm, ahead of the
LDS-DMA of the context tiles, and wait for them with an asm `s_waitcnt` that
takes the destination registers as operands.  Correctness then rests on the
register allocator never reading (or copying) those registers between the
load and that wait: the data lands there asynchronously.  This test compiles
decode_step.hip for gfx950 with the library's flags and scans every kernel
for such an early read.  CPU only (hipcc cross-compiles).

The tile DMAs are inline asm too (global_load_lds_dwordx4 with an SGPR base).
The compiler cannot see the SGPR read inside the asm, so it does not insert
the five wait states the hardware needs after a vector instruction writes
those SGPRs; a base moved there by v_readfirstlane just before the asm was
read stale and sent a tile DMA to a wild address.  The asm therefore waits
them out itself (s_nop 4); the DMA tests check that every SGPR-base DMA of
the kernel sources (and of the streaming-ceiling program) does, and that
no base is left in VGPRs."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2609_05707_amd import build as B


def _vregs(tok: str) -> set:
    out = set()
    for m in re.finditer(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b", tok):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


_TERMINATORS = ("s_branch", "s_endpgm", "s_setpc_b64")


def _blocks(lines):
    """Split a kernel body into basic blocks [label, instructions, successors]:
    a block ends at a label or after any branch (a conditional branch falls
    through to the next block)."""
    blocks, cur, label = [], [], None
    for line in lines:
        raw = line.strip()
        t = raw if raw.startswith(";;#ASM") else raw.split(";")[0].strip()
        m = re.match(r"^(\.LBB\w+):", t)
        if m:
            blocks.append([label, cur])
            label, cur = m.group(1), []
            continue
        if not t or t.startswith("."):
            continue
        cur.append(t)
        if t.startswith(("s_branch", "s_cbranch", "s_endpgm", "s_setpc_b64")):
            blocks.append([label, cur])
            label, cur = None, []
    blocks.append([label, cur])
    out = []
    for k, (lab, ins) in enumerate(blocks):
        succ = []
        last = ins[-1].split()[0] if ins else ""
        if last.startswith(("s_branch", "s_cbranch")):
            succ.append(ins[-1].split()[1])
        if last not in _TERMINATORS and k + 1 < len(blocks):
            succ.append(("#next", k + 1))
        out.append((lab, ins, succ))
    return out


def early_reads(asm: str):
    """(kernel, instruction) of every instruction that reads or overwrites a
    register that an asm global load may not yet have delivered: a forward
    dataflow over the kernel's basic blocks, where a load's destination
    stays pending until an asm s_waitcnt (the tied wait) or a compiler
    s_waitcnt vmcnt(0)."""
    hits = []
    for name in re.findall(r"^(_ZN4ippd\w+):", asm, re.M):
        a = asm.index(name + ":")
        b = asm.index(".Lfunc_end", a)
        blocks = _blocks(asm[a:b].splitlines()[1:])
        index = {lab: k for k, (lab, _, _) in enumerate(blocks) if lab}
        succs = [[index[s] if not isinstance(s, tuple) else s[1] for s in sl if isinstance(s, tuple) or s in index]
                 for _, _, sl in blocks]
        state_in = [None] * len(blocks)
        state_in[0] = frozenset()
        work = [0]
        found = {}
        while work:
            k = work.pop()
            pending, in_asm = set(state_in[k]), False
            for t in blocks[k][1]:
                if t.startswith(";;#ASMSTART"):
                    in_asm = True
                    continue
                if t.startswith(";;#ASMEND"):
                    in_asm = False
                    continue
                op = t.split()[0]
                if in_asm and op.startswith("global_load") and "lds" not in op:
                    pending |= _vregs(t.split()[1].rstrip(","))
                    continue
                if op == "s_waitcnt" and (in_asm or re.search(r"vmcnt\(0\)", t)):
                    pending = set()
                    continue
                if not pending or op.startswith("s_"):
                    continue
                fields = [f.strip() for f in t.split(None, 1)[1].split(",")] if " " in t else []
                srcs = set()
                for f in fields[1:]:
                    srcs |= _vregs(f)
                dst = _vregs(fields[0]) if fields else set()
                if op.startswith(("global_store", "ds_write", "buffer_store", "scratch_store")):
                    srcs |= dst
                    dst = set()
                if srcs & pending or dst & pending:
                    found[(name, t)] = True
                pending -= dst
            out = frozenset(pending)
            for sk in succs[k]:
                new = out if state_in[sk] is None else state_in[sk] | out
                if new != state_in[sk]:
                    state_in[sk] = new
                    work.append(sk)
        hits += list(found)
    return hits


def test_scanner_flags_a_planted_copy():
    asm = "\n".join([
        "_ZN4ippd1kEv:",
        "s_nop 0",
        ";;#ASMSTART", "global_load_dwordx4 v[2:5], v[8:9], off", ";;#ASMEND",
        "v_mov_b32_e32 v10, v3",
        ";;#ASMSTART", "s_waitcnt vmcnt(0)", ";;#ASMEND",
        ".Lfunc_end0:",
    ])
    assert len(early_reads(asm)) == 1
    clean = asm.replace("v_mov_b32_e32 v10, v3", "v_mov_b32_e32 v10, v7")
    assert early_reads(clean) == []


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_no_early_reads_of_asm_loads(tmp_path):
    out = tmp_path / "decode_step.s"
    flags = [f for f in B.flags_for("decode_step.hip") if f != "-fPIC"]
    cmd = [B.hipcc(), *flags, "--cuda-device-only", "-S", os.path.join(B.CSRC, "decode_step.hip"), "-o", str(out)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    asm = out.read_text()
    assert "global_load_lds_dwordx4" in asm and ";;#ASMSTART" in asm
    hits = early_reads(asm)
    assert hits == [], hits[:10]
    assert dma_hazards(asm) == []


def dma_hazards(asm: str):
    """SGPR-base LDS-DMAs of an assembly listing that are not preceded, in
    their own asm block, by s_nop 4 (or whose base operand is a VGPR)."""
    bad = []
    lines = [line.strip() for line in asm.splitlines()]
    for k, t in enumerate(lines):
        if not t.startswith("global_load_lds_dwordx4"):
            continue
        ops = [f.strip() for f in t.split(None, 1)[1].split(",")]
        if len(ops) < 2 or ops[1] == "off":
            continue                                  # per-lane 64-bit address form
        if not ops[1].startswith("s["):
            bad.append(("vgpr base", t))
            continue
        if k == 0 or lines[k - 1] != "s_nop 4":
            bad.append(("no wait states", t))
    return bad


def test_dma_hazard_scan_flags_planted_cases():
    ok = "\n".join([";;#ASMSTART", "s_nop 4", "global_load_lds_dwordx4 v3, s[4:5]", ";;#ASMEND"])
    assert dma_hazards(ok) == []
    assert len(dma_hazards(ok.replace("s_nop 4", "s_nop 0"))) == 1
    assert len(dma_hazards(ok.replace("s[4:5]", "v[4:5]"))) == 1
    per_lane = "\n".join([";;#ASMSTART", "s_nop 0", "global_load_lds_dwordx4 v[2:3], off", ";;#ASMEND"])
    assert dma_hazards(per_lane) == []


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
@pytest.mark.parametrize("src", ["prefill.hip", "dense_mask.hip", "stream_ceiling.hip"])
def test_dma_bases_in_sgprs_with_wait_states(tmp_path, src):
    out = tmp_path / (src + ".s")
    flags = [f for f in B.flags_for(src) if f != "-fPIC"]
    cmd = [B.hipcc(), *flags, "--cuda-device-only", "-S", os.path.join(B.CSRC, src), "-o", str(out)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    asm = out.read_text()
    assert "global_load_lds_dwordx4" in asm
    assert dma_hazards(asm) == []
