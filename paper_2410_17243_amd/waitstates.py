"""Wait-state check of the inline-assembly MFMA and DMA instructions.

The compiler inserts the wait states that gfx950 requires between dependent
instructions it generates itself, but it does not look inside inline assembly.
The kernels issue two kinds of instructions from inline assembly:

  * the LDS DMA ``buffer_load_dwordx4 ... lds``, whose address VGPR,
    descriptor SGPRs, offset SGPR and m0 the compiler may set up (or restore
    with ``v_readlane`` / ``v_accvgpr_read``) right before the statement;
  * chains of ``v_mfma_*`` whose source operands the compiler may restore with
    a VALU instruction right before the statement, and whose accumulator the
    compiler could copy or spill between two links of a chain.

Each such statement carries its own ``s_nop`` padding.  This module checks the
padding against the generated code, so that a change in the sources or in the
compiler that breaks it is caught on the CPU before anything runs on a GPU:

  1. between the last VALU write of any source register of an inline-asm MFMA
     and the MFMA: at least ``MFMA_SRC_WAIT`` wait states;
  2. between the last VALU write of any SGPR, VGPR or m0 that an inline-asm
     DMA reads and the DMA: at least ``DMA_SRC_WAIT`` wait states (a VALU
     write of an SGPR read by a vector-memory instruction needs five), and at
     least one after a scalar write of m0;
  3. after an inline-asm MFMA, no instruction other than another MFMA that
     accumulates into the same registers may read or write its result
     registers within ``MFMA_RESULT_WAIT`` wait states (the result of a 32x32
     MFMA is not readable before then).

Wait states are counted as issue slots: one per instruction, N + 1 for
``s_nop N``.  The search follows branches backwards (every branch into a
label) and forwards (branch targets and fall-through), so a block entered from
elsewhere is checked along each path.

    python -m paper_2410_17243_amd.waitstates file.s [...]   # scan assembly
"""

from __future__ import annotations

import re
import sys
from dataclasses import dataclass

MFMA_SRC_WAIT = 2
DMA_SRC_WAIT = 5
DMA_M0_SALU_WAIT = 1
MFMA_RESULT_WAIT = 18

_REG = re.compile(r"\b([vas])\[(\d+):(\d+)\]|\b([vas])(\d+)\b|\b(m0)\b")
_LABEL = re.compile(r"^([.\w$]+):")
_FUNC = re.compile(r"^([_A-Za-z][\w.$]*):\s*(;.*)?$")


@dataclass
class Inst:
    text: str       # the instruction without comments
    op: str         # mnemonic
    inline: bool    # inside an inline-asm region
    line: int       # 1-based line in the assembly file


@dataclass
class Violation:
    func: str
    line: int
    inst: str
    rule: str
    other: str
    waits: int

    def __str__(self):
        return f"{self.func}: line {self.line}: '{self.inst}' {self.rule} ('{self.other}' {self.waits} wait states away)"


def regs_of(operands: str) -> set:
    """Registers named in an operand string, as 'v12', 'a3', 's40', 'm0'."""
    out = set()
    for m in _REG.finditer(operands):
        if m.group(1):
            out.update(f"{m.group(1)}{r}" for r in range(int(m.group(2)), int(m.group(3)) + 1))
        elif m.group(4):
            out.add(f"{m.group(4)}{m.group(5)}")
        else:
            out.add("m0")
    return out


def _split_operands(text: str):
    parts = text.split(None, 1)
    if len(parts) < 2:
        return []
    ops, depth, cur = [], 0, ""
    for ch in parts[1]:
        if ch == "[":
            depth += 1
        elif ch == "]":
            depth -= 1
        if ch == "," and depth == 0:
            ops.append(cur.strip())
            cur = ""
        else:
            cur += ch
    if cur.strip():
        ops.append(cur.strip())
    return ops


def waits_of(inst: Inst) -> int:
    if inst.op == "s_nop":
        m = re.search(r"s_nop\s+(0x[0-9a-fA-F]+|\d+)", inst.text)
        return int(m.group(1), 0) + 1 if m else 1
    return 1


def is_valu(op: str) -> bool:
    return op.startswith("v_") and not op.startswith(("v_mfma", "v_smfmac"))


def is_mfma(op: str) -> bool:
    return op.startswith(("v_mfma", "v_smfmac"))


def is_dma(inst: Inst) -> bool:
    return inst.op.startswith("buffer_load") and re.search(r"\blds\b", inst.text) is not None


def written_by(inst: Inst) -> set:
    """Registers an instruction writes (its first operand for VALU, SALU and
    loads; m0 for an s_mov to m0)."""
    ops = _split_operands(inst.text)
    if not ops:
        return set()
    if inst.op.startswith(("s_", "v_", "ds_read", "ds_load", "buffer_load", "global_load", "flat_load",
                           "scratch_load")):
        if inst.op.startswith(("s_nop", "s_wait", "s_barrier", "s_cbranch", "s_branch", "s_set", "s_endpgm",
                               "s_sleep", "s_sendmsg", "s_trap", "s_icache")):
            return set()
        if is_dma(inst):
            return set()
        return regs_of(ops[0])
    return set()


def mfma_sources(inst: Inst) -> set:
    ops = _split_operands(inst.text)
    out = set()
    for o in ops[1:4]:
        out |= regs_of(o)
    return out


def mfma_dest(inst: Inst) -> set:
    ops = _split_operands(inst.text)
    return regs_of(ops[0]) if ops else set()


def dma_sources(inst: Inst) -> set:
    ops = _split_operands(inst.text)
    out = {"m0"}
    for o in ops[:3]:
        out |= regs_of(o)
    return out


def parse(text: str):
    """Functions of an assembly file: name -> (instructions, labels, branches)."""
    funcs = {}
    cur = None
    inline = False
    for ln_no, raw in enumerate(text.split("\n"), 1):
        line = raw.split(";;")[0] if not raw.strip().startswith(";;#ASM") else raw
        s = raw.strip()
        if s.startswith(";;#ASMSTART"):
            inline = True
            continue
        if s.startswith(";;#ASMEND"):
            inline = False
            continue
        if not s or s.startswith(";") or s.startswith("//"):
            continue
        m = _FUNC.match(s)
        if m and not s.startswith("."):
            cur = m.group(1)
            funcs[cur] = {"insts": [], "labels": {}, "entries": []}
            continue
        if cur is None:
            continue
        m = _LABEL.match(s)
        if m:
            funcs[cur]["labels"][m.group(1)] = len(funcs[cur]["entries"])
            funcs[cur]["entries"].append(("label", m.group(1)))
            continue
        if s.startswith("."):
            continue
        body = line.split(";")[0].strip()
        if not body:
            continue
        op = body.split()[0]
        funcs[cur]["entries"].append(("inst", Inst(body, op, inline, ln_no)))
    for f in funcs.values():
        branches = {}
        for idx, (kind, e) in enumerate(f["entries"]):
            if kind == "inst" and (e.op.startswith("s_cbranch") or e.op == "s_branch"):
                tgt = e.text.split()[-1]
                branches.setdefault(tgt, []).append(idx)
        f["branches"] = branches
    return funcs


def _unconditional(e) -> bool:
    return e[0] == "inst" and e[1].op in ("s_branch", "s_endpgm", "s_setpc_b64")


def _lookback(f, start: int, need: int, pred, limit: int = 4096):
    """Smallest wait-state distance from entry `start` back to an instruction
    matching pred (None if none within `need`), over all incoming paths."""
    entries, labels, branches = f["entries"], f["labels"], f["branches"]
    best = [None]
    seen = {}
    stack = [(start - 1, 0)]
    steps = 0
    while stack and steps < limit:
        idx, ws = stack.pop()
        steps += 1
        while idx >= 0 and ws < need:
            if seen.get(idx, need + 1) <= ws:
                break
            seen[idx] = ws
            kind, e = entries[idx]
            if kind == "label":
                for b in branches.get(e, []):
                    stack.append((b, ws))
                if idx > 0 and _unconditional(entries[idx - 1]):
                    break
                idx -= 1
                continue
            if pred(e):
                if best[0] is None or ws < best[0][0]:
                    best[0] = (ws, e)
                break
            ws += waits_of(e)
            idx -= 1
    return best[0]


def _lookahead(f, start: int, need: int, pred, stop, limit: int = 4096):
    """First instruction matching pred within `need` wait states after entry
    `start` on any outgoing path, unless `stop` matches first."""
    entries, labels = f["entries"], f["labels"]
    seen = {}
    stack = [(start + 1, 0)]
    steps = 0
    found = None
    while stack and steps < limit:
        idx, ws = stack.pop()
        steps += 1
        while idx < len(entries) and ws < need:
            if seen.get(idx, need + 1) <= ws:
                break
            seen[idx] = ws
            kind, e = entries[idx]
            if kind == "label":
                idx += 1
                continue
            if stop(e):
                break
            if pred(e):
                if found is None or ws < found[0]:
                    found = (ws, e)
                break
            if e.op.startswith("s_cbranch") or e.op == "s_branch":
                tgt = e.text.split()[-1]
                if tgt in labels:
                    stack.append((labels[tgt], ws + 1))
                if e.op == "s_branch":
                    break
            if e.op in ("s_endpgm", "s_setpc_b64"):
                break
            ws += waits_of(e)
            idx += 1
    return found


def scan(text: str):
    """All violations of rules 1-3 in one assembly file, and the number of
    inline-asm MFMA and DMA instructions checked."""
    out = []
    checked = 0
    for fname, f in parse(text).items():
        for idx, (kind, e) in enumerate(f["entries"]):
            if kind != "inst" or not e.inline:
                continue
            if is_mfma(e.op):
                checked += 1
                srcs = mfma_sources(e)
                hit = _lookback(f, idx, MFMA_SRC_WAIT, lambda x: is_valu(x.op) and bool(written_by(x) & srcs))
                if hit:
                    out.append(Violation(fname, e.line, e.text, "reads a register a VALU instruction wrote too recently",
                                         hit[1].text, hit[0]))
                dst = mfma_dest(e)
                size = len(dst)

                def chained(x, dst=dst, size=size):
                    return is_mfma(x.op) and x.inline and mfma_dest(x) == dst and len(mfma_sources(x) & dst) == size

                hit = _lookahead(f, idx, MFMA_RESULT_WAIT,
                                 lambda x: not chained(x) and bool((written_by(x) | _read_regs(x)) & dst),
                                 stop=chained)
                if hit:
                    out.append(Violation(fname, e.line, e.text, "result touched before it is ready", hit[1].text,
                                         hit[0]))
            elif is_dma(e):
                checked += 1
                srcs = dma_sources(e)
                hit = _lookback(f, idx, DMA_SRC_WAIT, lambda x: is_valu(x.op) and bool(written_by(x) & srcs))
                if hit:
                    out.append(Violation(fname, e.line, e.text, "reads a register a VALU instruction wrote too recently",
                                         hit[1].text, hit[0]))
                hit = _lookback(f, idx, DMA_M0_SALU_WAIT, lambda x: x.op.startswith("s_") and "m0" in written_by(x))
                if hit:
                    out.append(Violation(fname, e.line, e.text, "m0 written too recently", hit[1].text, hit[0]))
    return out, checked


def _read_regs(inst: Inst) -> set:
    ops = _split_operands(inst.text)
    out = set()
    for o in ops[1:]:
        out |= regs_of(o)
    if inst.op.startswith(("ds_write", "ds_store", "buffer_store", "global_store", "scratch_store", "flat_store")):
        out |= regs_of(ops[0]) if ops else set()
    return out


def main(argv):
    total = 0
    bad = 0
    for path in argv:
        v, n = scan(open(path).read())
        total += n
        bad += len(v)
        for x in v[:20]:
            print(f"{path}: {x}")
    print(f"checked {total} inline-asm MFMA/DMA instructions: {bad} violations")
    return 1 if bad else 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
