"""Build-time check of the generated gfx950 assembly for matrix-core results
read too early.

A branch around an MFMA whose accumulator is read after the join was once
compiled without the wait states that the read needs, which gave wrong and
non-deterministic results.  The kernels therefore issue every MFMA
unconditionally, and this check scans the device assembly of each build:
after every v_mfma it walks the following instructions (counting one state
per instruction, N + 1 per s_nop N, up to an unconditional branch) and
reports the first instruction that
reads one of the MFMA's destination registers with fewer states in between
than the instruction's threshold, or another MFMA that takes them as its A
or B operand (its C operand may chain: the hardware forwards it).

The thresholds are per instruction: the fewest states the compiler itself
leaves after that MFMA before a read on any straight-line path of this
library (8 after the 16-bit 16x16x32 forms, 10 after the fp32 16x16x4), so a
path that lost them, as in the miscompilation above, is reported.  It is a
guard against that failure, not a hazard model of the hardware: the
determinism tests (repeated runs, the one-launch kernels against the
chain byte for byte, graph replays) are the check of the results.
"""
from __future__ import annotations

import re

MIN_STATES = {
    "v_mfma_f32_16x16x32_f16": 8,
    "v_mfma_f32_16x16x32_bf16": 8,
    "v_mfma_f32_16x16x4_f32": 10,
}
DEFAULT_STATES = 4  # any other MFMA form
WINDOW = 60

_RANGE = re.compile(r"([av])\[(\d+):(\d+)\]")
_SINGLE = re.compile(r"([av])(\d+)$")


def _regs(op: str) -> set:
    m = _RANGE.match(op)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = _SINGLE.match(op)
    if m:
        return {(m.group(1), int(m.group(2)))}
    return set()


def _operands(text: str) -> list:
    return [o.strip() for o in text.split(",")]


def check(asm: str) -> list:
    """Findings (strings) for the assembly text; empty when clean."""
    lines = asm.splitlines()
    found = []
    func = "?"
    for i, line in enumerate(lines):
        if re.match(r"^_Z\w+:", line):
            func = line.split(":")[0]
        s = line.strip()
        if not s.startswith("v_mfma"):
            continue
        name, rest = s.split(None, 1)
        need = MIN_STATES.get(name, DEFAULT_STATES)
        ops = _operands(rest)
        dst = _regs(ops[0])
        states = 0
        for j in range(i + 1, min(i + WINDOW, len(lines))):
            t = lines[j].strip()
            if not t or t.startswith((";", ".")) or t.endswith(":"):
                continue
            parts = t.split(None, 1)
            op = parts[0]
            if op in ("s_branch", "s_endpgm", "s_setpc_b64"):
                break  # the text that follows is not this path's next instruction
            if op.startswith("s_nop"):
                states += int(parts[1].split()[0], 0) + 1
                continue
            args = _operands(parts[1]) if len(parts) > 1 else []
            if op.startswith("v_mfma"):
                if any(_regs(a) & dst for a in args[1:3]):
                    found.append("%s: MFMA A/B operand reads a pending MFMA result: %s" % (func, t))
                states += 1
                continue
            reads = set()
            srcs = args if op.startswith(("global_store", "ds_write", "buffer_store", "flat_store")) else args[1:]
            for a in srcs:
                reads |= _regs(a)
            if reads & dst:
                if states < need:
                    found.append("%s: MFMA result read after %d states: %s" % (func, states, t))
                break
            if dst & _regs(args[0] if args else ""):
                break  # destination overwritten first
            states += 1
    return found
