"""Wait-state check of the hand-written assembly blocks in the indexer kernels.

The indexer's MFMA + epilogue groups are inline assembly, and the compiler
inserts no wait states inside them (nor before a read of an MFMA result in
them).  The blocks therefore carry their own s_nop padding, counted by the
rules their comments state:

  * a read of an 8-pass MFMA result (v_mfma_scale_f32_16x16x128_f8f6f4)
    comes at least 12 wait states after the MFMA, where each later 8-pass
    MFMA counts as 4, an s_nop N as N + 1 and any other instruction as 1;
  * a read of a 4-pass MFMA result (v_mfma_f32_16x16x32_bf16) comes at least
    8 wait states after it, except by the next MFMA of the same kind
    accumulating into exactly those registers (back to back), and the end of
    the block (after which anything may read it) comes at least 8 after;
  * an MFMA reads a register written by a VALU instruction at least 2 wait
    states after the write, and the first MFMA of a block comes at least 2
    wait states after the block's start (a VALU write of one of its sources
    may precede the block);
  * a read of a register written by another VALU instruction of the block
    comes at least 1 wait state later, except a v_dot2c accumulating into
    the register the previous v_dot2c wrote;
  * an instruction other than a v_dot2c that reads a v_dot2c result, and the
    end of the block, come at least 3 wait states after the last v_dot2c.

This module parses the compiled assembly (`hipcc -S`) and reports every
instruction that breaks one of the rules.  It knows only the instructions
those blocks use.
"""
import re

MFMA_REQ = 12        # wait states from an 8-pass MFMA to a read of its result
MFMA_COUNT = 4       # what a later 8-pass MFMA counts for
MFMA4_REQ = 8        # 4-pass MFMA -> a read of its result other than an accumulation, and block end
VALU_REQ = 1         # VALU write -> read by another VALU instruction
VALU_MFMA_REQ = 2    # VALU write -> read by an MFMA
DOT_REQ = 3          # v_dot2c result -> any other reader, and block end
START_REQ = 2        # block start -> first MFMA
MFMA8_OPS = ("v_mfma_scale_f32_16x16x128_f8f6f4",)
MFMA4_OPS = ("v_mfma_f32_16x16x32_bf16",)

_REG = re.compile(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b")


def _regs(text):
    out = set()
    for m in _REG.finditer(text):
        if m.group(1) is not None:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
        else:
            out.add(int(m.group(3)))
    return out


def _parse(line):
    """(opcode, destination registers, source registers, accumulator registers) of one line;
    the accumulator is the MFMA source C when it is exactly the destination."""
    line = line.split(";")[0].strip()
    if not line:
        return None
    op, _, rest = line.partition(" ")
    ops = [o.strip() for o in re.split(r",(?![^\[]*\])", rest) if o.strip()]
    if op.startswith("s_"):
        return op, set(), set(), set()
    dst = _regs(ops[0]) if ops else set()
    src = set()
    for o in ops[1:]:
        src |= _regs(o.split(" ")[0])
    acc = set()
    if op.startswith("v_mfma") and len(ops) >= 4 and _regs(ops[3].split(" ")[0]) == dst:
        acc = dst
    if op.startswith("v_dot2c"):
        src |= dst  # accumulates into its destination
    return op, dst, src, acc


def _kind(op):
    if op in MFMA8_OPS:
        return "mfma"
    if op in MFMA4_OPS:
        return "mfma4"
    if op.startswith("v_mfma"):
        raise ValueError(f"unknown MFMA {op}")
    return "dot" if op.startswith("v_dot2c") else "valu"


def _cost(op, line):
    if op == "s_nop":
        return int(line.split()[1]) + 1
    if op in MFMA8_OPS:
        return MFMA_COUNT
    return 1


def blocks(asm_text):
    """The inline assembly blocks of a compiled .s file, as lists of lines."""
    out, cur = [], None
    for line in asm_text.splitlines():
        s = line.strip()
        if s.startswith(";;#ASMSTART"):
            cur = []
        elif s.startswith(";;#ASMEND"):
            if cur is not None:
                out.append(cur)
            cur = None
        elif cur is not None and s and not s.startswith(";"):
            cur.append(s)
    return out


def check_block(lines):
    """Violations of the rules in one block, as strings (empty: none)."""
    bad = []
    # per register: (kind, position in wait states at which it was written)
    written = {}
    t = 0             # wait states elapsed before the current instruction
    seen_mfma = False
    for line in lines:
        p = _parse(line)
        if p is None:
            continue
        op, dst, src, acc = p
        is_mfma = op.startswith("v_mfma")
        kind_here = _kind(op) if op.startswith("v_") else None
        if is_mfma and not seen_mfma:
            seen_mfma = True
            if t < START_REQ:
                bad.append(f"{line}: first MFMA {t} wait states after the block start (< {START_REQ})")
        for r in src:
            if r not in written:
                continue
            kind, tw = written[r]
            dist = t - tw
            if kind == "mfma":
                need = MFMA_REQ
            elif kind == "mfma4":
                # the next MFMA of the same kind accumulating into exactly these registers needs none
                need = 0 if (kind_here == "mfma4" and r in acc) else MFMA4_REQ
            elif is_mfma:
                need = VALU_MFMA_REQ
            elif kind == "dot":
                # a v_dot2c accumulating into a v_dot2c result needs none
                need = 0 if (op.startswith("v_dot2c") and r in dst) else DOT_REQ
            else:
                need = VALU_REQ
            if dist < need:
                bad.append(f"{line}: reads v{r} {dist} wait states after its {kind} write (< {need})")
        cost = _cost(op, line)
        if op.startswith("v_"):
            # the result is readable from the instruction after this one: a
            # read right behind it is 0 wait states away
            for r in dst:
                written[r] = (kind_here, t + cost)
        t += cost
    for r, (kind, tw) in written.items():
        if kind == "dot" and t - tw < DOT_REQ:
            bad.append(f"block end: v{r} {t - tw} wait states after its v_dot2c write (< {DOT_REQ})")
        if kind == "mfma4" and t - tw < MFMA4_REQ:
            bad.append(f"block end: v{r} {t - tw} wait states after its 4-pass MFMA write (< {MFMA4_REQ})")
    return bad
