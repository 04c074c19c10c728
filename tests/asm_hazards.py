"""Static checks of the hand-placed matrix-core instructions in device assembly.

The kernels issue some MFMAs as inline asm so that every operand stays in the
register file the kernel chose.  The compiler does not treat such an asm
statement as an MFMA, so it neither inserts the wait states an MFMA needs
around its sources nor keeps an MFMA's accumulator input alive while the
matrix core still reads it.  Two rules are checked on the compiler's
assembly output (CDNA3/CDNA4 ISA, dependency-resolution rules for MFMA):

  * a VALU instruction that writes a source register of an inline-asm MFMA
    needs at least two wait states before the MFMA (``s_nop N`` gives N + 1,
    any other instruction one);
  * an inline-asm MFMA whose accumulator input is a register range other than
    its output must not see that range written by any instruction among the
    next ``war_window`` instructions (the matrix core reads the accumulator
    input during its later passes).

The scan is textual: it follows the listing across labels and branches, so
it checks the straight-line order the compiler emitted.
"""
import re

_RANGE = re.compile(r"\b([va])\[(\d+):(\d+)\]|\b([va])(\d+)\b")


def _regs(text):
    out = set()
    for m in _RANGE.finditer(text):
        if m.group(1):
            out |= {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
        else:
            out.add((m.group(4), int(m.group(5))))
    return out


def _instructions(asm_text):
    """(line number, function, text, in inline asm) for every instruction."""
    func, in_asm = None, False
    for n, line in enumerate(asm_text.split("\n"), 1):
        s = line.strip()
        if re.match(r"^[A-Za-z_.$][\w.$]*:", line) and not line.startswith((" ", "\t")):
            if not line.startswith("."):
                func = line.split(":")[0]
            continue
        if s.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if s.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if not s or s.startswith((";", ".")):
            continue
        yield n, func, s.split(";")[0].strip(), in_asm


def _operands(text):
    parts = text.split(None, 1)
    return parts[0], ([o.strip() for o in parts[1].split(",")] if len(parts) > 1 else [])


def check(asm_text, war_window=40):
    """Return a list of violation descriptions (empty when both rules hold)."""
    ins = [i for i in _instructions(asm_text) if i[2]]
    bad = []
    for k, (line, func, text, in_asm) in enumerate(ins):
        op, ops = _operands(text)
        if not (in_asm and op.startswith("v_mfma")) or len(ops) < 4:
            continue
        dst, srcc = _regs(ops[0]), _regs(ops[3])
        sources = _regs(",".join(ops[1:]))
        # Rule 1: VALU writes of a source, fewer than two wait states before.
        waits = 0
        for p in range(k - 1, -1, -1):
            if waits >= 2:
                break
            pop, pops = _operands(ins[p][2])
            if pop == "s_nop":
                waits += int(pops[0], 0) + 1
                continue
            if pop.startswith("v_") and not pop.startswith("v_mfma") and pops:
                if _regs(pops[0]) & sources:
                    bad.append(f"{func}: line {ins[p][0]} '{ins[p][2]}' writes a source of "
                               f"the MFMA at line {line} with {waits} wait states between")
            waits += 1
        # Rule 2: writes of a separate accumulator input while it is read.
        if srcc and not (srcc & dst):
            for q in range(k + 1, min(len(ins), k + 1 + war_window)):
                qop, qops = _operands(ins[q][2])
                if qop.startswith(("s_", "buffer_store", "global_store", "ds_write",
                                   "scratch_store")) or not qops:
                    continue
                if _regs(qops[0]) & srcc:
                    bad.append(f"{func}: line {ins[q][0]} '{ins[q][2]}' overwrites the "
                               f"accumulator input of the MFMA at line {line}")
    return bad
