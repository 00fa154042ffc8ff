"""Static check of the prefill kernels' machine code for MFMA data hazards.

The prefill kernel issues its MFMAs as inline assembly (to fix which register
file holds each operand), so the compiler does not insert the wait states that
gfx950 requires around them.  This test scans the device assembly that
build() keeps for every instantiation and follows the control flow from each
producer, counting wait states as the hardware rules do (s_nop N gives N + 1,
every other instruction 1):

  R1  a VALU write of a VGPR/AGPR, then an MFMA reading it: >= 2 wait states;
  R2  an MFMA result, then any other instruction reading or writing those
      registers (or another MFMA reading them as A/B, or as C without being
      the same accumulator chain): >= 20 wait states (the largest XDL
      requirement on gfx950 is 19, for 16-pass instructions);
  R3  an MFMA reading C, then a non-MFMA write of those registers: >= 16.

It needs no GPU.  If the assembly is missing or older than the sources, the
library is rebuilt first (about a minute).
"""

import os
import re

import pytest

from paper_2510_08726_amd import build as libbuild

CSRC = libbuild.CSRC
SOURCES = ["prefill.hip", "kernel_common.h", "launch.h"]

REG = re.compile(r"\b([va])(?:\[(0x[0-9a-fA-F]+|\d+)(?::(0x[0-9a-fA-F]+|\d+))?\]|(\d+)\b)")
R1_WAIT, R2_WAIT, R3_WAIT = 2, 20, 16


def _num(s):
    return int(s, 16) if s.startswith("0x") else int(s)


def regs(text):
    out = set()
    for m in REG.finditer(text):
        kind = m.group(1)
        if m.group(4) is not None:
            out.add((kind, int(m.group(4))))
        else:
            lo = _num(m.group(2))
            hi = _num(m.group(3)) if m.group(3) is not None else lo
            out.update((kind, r) for r in range(lo, hi + 1))
    return out


class Inst:
    __slots__ = ("op", "text", "defs", "uses", "srcc", "mfma", "valu", "wait", "target", "cond", "end")

    def __init__(self, text):
        self.text = text
        parts = text.split(None, 1)
        self.op = parts[0]
        ops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
        self.defs, self.uses, self.srcc = set(), set(), set()
        self.mfma = self.op.startswith("v_mfma")
        self.valu = self.op.startswith("v_") and not self.mfma
        self.wait = _num(ops[0]) + 1 if self.op == "s_nop" else 1
        self.target = ops[0] if self.op.startswith(("s_branch", "s_cbranch")) and ops else None
        self.cond = self.op.startswith("s_cbranch")
        self.end = self.op == "s_endpgm"
        op = self.op
        if self.mfma:
            self.defs = regs(ops[0])
            self.uses = regs(",".join(ops[1:]))
            self.srcc = regs(ops[3]) if len(ops) > 3 else set()
        elif op.startswith(("v_cmp", "v_readfirstlane", "v_readlane")):
            self.uses = regs(",".join(ops[1:]))
        elif op.startswith(("v_permlane16_swap", "v_permlane32_swap")):
            self.defs = regs(",".join(ops[:2]))
            self.uses = set(self.defs)
        elif op.startswith("v_"):
            self.defs = regs(ops[0]) if ops else set()
            self.uses = regs(",".join(ops[1:]))
        elif op.startswith(("ds_read", "ds_load", "ds_bpermute", "ds_permute", "ds_swizzle")):
            self.defs = regs(ops[0])
            self.uses = regs(",".join(ops[1:]))
        elif op.startswith(("buffer_load", "global_load", "scratch_load", "flat_load")):
            if "lds" in ops:
                self.uses = regs(",".join(ops))
            else:
                self.defs = regs(ops[0])
                self.uses = regs(",".join(ops[1:]))
        elif op.startswith(("ds_", "buffer_", "global_", "scratch_", "flat_")):
            self.uses = regs(",".join(ops))


def kernels(path):
    """{kernel name: (instructions, label -> index)} of one assembly file."""
    out = {}
    name, insts, labels = None, [], {}
    for raw in open(path):
        line = raw.split(";", 1)[0].split("//", 1)[0].strip()
        if not line:
            continue
        if line.endswith(":"):
            lab = line[:-1]
            if lab.startswith("_Z") and "prefill_kernel" in lab:
                name, insts, labels = lab, [], {}
                out[name] = (insts, labels)
            elif name is not None:
                labels[lab] = len(insts)
            continue
        if name is None or line.startswith("."):
            continue
        for piece in line.split("\n"):
            if piece.strip():
                insts.append(Inst(piece.strip()))
    return out


def successors(insts, labels, i):
    ins = insts[i]
    if ins.end:
        return []
    if ins.target is not None:
        tgt = [labels[ins.target]] if ins.target in labels else []
        return tgt + ([i + 1] if ins.cond and i + 1 < len(insts) else [])
    return [i + 1] if i + 1 < len(insts) else []


def scan(insts, labels, start, budget, hit):
    """Visit every instruction reachable from `start` (exclusive) with fewer
    than `budget` wait states in between; hit(inst, waits) -> message or None."""
    found = []
    seen = set()
    stack = [(j, 0) for j in successors(insts, labels, start)]
    while stack:
        j, w = stack.pop()
        if w >= budget or (j, w) in seen:
            continue
        seen.add((j, w))
        msg = hit(insts[j], w)
        if msg:
            found.append(msg)
        stack.extend((k, w + insts[j].wait) for k in successors(insts, labels, j))
    return found


def check_kernel(insts, labels):
    problems = []
    for i, p in enumerate(insts):
        if p.valu and p.defs:
            d = p.defs

            def r1(q, w, d=d, p=p):
                if q.mfma and q.uses & d:
                    return f"R1 {w} wait states: '{p.text}' -> '{q.text}'"
            problems += scan(insts, labels, i, R1_WAIT, r1)
        if p.mfma:
            d = p.defs

            def r2(q, w, d=d, p=p):
                if q.mfma:
                    chain = q.srcc == d and q.defs == d
                    a_b = q.uses - q.srcc
                    if (a_b & d) or (q.srcc & d and not chain):
                        return f"R2 {w} wait states: '{p.text}' -> '{q.text}'"
                elif (q.uses | q.defs) & d:
                    return f"R2 {w} wait states: '{p.text}' -> '{q.text}'"
            problems += scan(insts, labels, i, R2_WAIT, r2)
            c = p.srcc

            def r3(q, w, c=c, p=p):
                if not q.mfma and q.defs & c:
                    return f"R3 {w} wait states: '{p.text}' -> '{q.text}'"
            if c:
                problems += scan(insts, labels, i, R3_WAIT, r3)
    return problems


def fresh_asm():
    files = libbuild.prefill_asm_files()
    newest_src = max(os.path.getmtime(os.path.join(CSRC, s)) for s in SOURCES)
    if not all(os.path.exists(f) and os.path.getmtime(f) >= newest_src for f in files):
        libbuild.build()
    return files


def test_regs_parser():
    assert regs("a[0x80:0x83]") == {("a", r) for r in range(128, 132)}
    assert regs("v[4:5], v7, a3") == {("v", 4), ("v", 5), ("v", 7), ("a", 3)}
    mf = Inst("v_mfma_f32_32x32x16_f16 a[0:15], v[4:7], v[8:11], a[0:15]")
    assert mf.mfma and ("a", 15) in mf.defs and mf.srcc == mf.defs


def test_checker_catches_planted_hazards():
    """The rules fire on the patterns they exist for."""
    mfma = "v_mfma_f32_32x32x16_f16 v[0:15], v[16:19], a[0:3], v[0:15]"
    bad_r1 = [Inst("v_mov_b32 v16, v40"), Inst(mfma), Inst("s_endpgm")]
    assert any(m.startswith("R1") for m in check_kernel(bad_r1, {}))
    bad_r2 = [Inst(mfma), Inst("s_nop 7"), Inst("v_add_f32 v40, v3, v41"), Inst("s_endpgm")]
    assert any(m.startswith("R2") for m in check_kernel(bad_r2, {}))
    ok = [Inst(mfma), Inst("s_nop 7"), Inst("s_nop 7"), Inst("s_nop 7"), Inst("v_add_f32 v40, v3, v41"),
          Inst("s_endpgm")]
    assert check_kernel(ok, {}) == []
    # across a loop back edge
    loop = [Inst("v_mov_b32 v17, v40"), Inst("s_cbranch_scc1 .LBB0_1"), Inst("s_endpgm")]
    body = [Inst(mfma)]
    insts = body + loop
    assert any(m.startswith("R1") for m in check_kernel(insts, {".LBB0_1": 0}))


def test_prefill_kernels_have_no_mfma_hazards():
    files = fresh_asm()
    nkern = 0
    problems = []
    for f in files:
        for name, (insts, labels) in kernels(f).items():
            nkern += 1
            assert sum(i.mfma for i in insts) > 0, name
            problems += [f"{name}: {m}" for m in check_kernel(insts, labels)]
    assert nkern == 32, nkern   # every prefill instantiation (see test_kernel_coverage)
    assert not problems, "\n".join(problems[:20]) + f"\n... {len(problems)} in total"
