"""Wait-state check of the gfx950 device assembly of this library.

The kernels issue their matrix products from inline asm, which the
compiler's hazard recognizer does not look into: a register copy or a VALU
write that the compiler places right before such a product, or a read of a
product's result placed right after it, gets no wait states from the
compiler.  The hardware does not interlock these cases; the product then
reads a stale operand, or the VALU reads a result not yet written.  This
module scans the assembly (hipcc --cuda-device-only -S) of every kernel,
follows branches, and reports each pair of instructions closer than the
matrix-core dependency rules of the CDNA3/CDNA4 instruction set allow:

  VALU write  -> MFMA read of that VGPR (SrcA, SrcB or SrcC):        2
  MFMA write  -> VALU / LDS / memory read or write of that VGPR:     P + 3
  MFMA write  -> MFMA read as SrcA / SrcB:                           P + 3
  MFMA write  -> MFMA read as SrcC, not the identical register range: P + 3
  MFMA SrcC   -> VALU write of that VGPR (write after read):         P - 1

(P = the product's passes, rounded up per shape: 8 for 16x16, 16 for
32x32, 2 for 4x4.)  A wait state is one issued instruction; `s_nop N`
counts N + 1.  Every figure is at or above what the instruction set asks
for, and products count one wait state however long they run, so the check
errs towards reporting.  Back-to-back accumulation into the same registers
(SrcC = vDst, same opcode) needs none.  Only pairs with at least one
instruction from inline asm are reported: the compiler resolves the others.
"""
import re
import sys

_REG = re.compile(r"\b([va])(?:(\d+)|\[(\d+):(\d+)\])")
_LABEL = re.compile(r"^([.\w$]+):")
_BRANCH = re.compile(r"^s_(?:cbranch_\w+|branch)\s+([.\w$]+)")
# VALU instructions that write both of their register operands
_WRITES_BOTH = ("v_swap_b32", "v_swap_b16", "v_permlane16_swap_b32", "v_permlane32_swap_b32")


def _passes(op):
    """Passes of a product, rounded up: 4x4 shapes 2, 16x16 shapes 8, 32x32
    shapes and anything not recognised 16."""
    m = re.match(r"v_mfma_\w*?(\d+)x(\d+)x(\d+)", op)
    if not m:
        return 16
    mm = int(m.group(1))
    return 2 if mm == 4 else 8 if mm == 16 else 16


def _regs(text):
    out = set()
    for kind, one, lo, hi in _REG.findall(text):
        if one:
            out.add((kind, int(one)))
        else:
            out.update((kind, r) for r in range(int(lo), int(hi) + 1))
    return out


class Ins:
    __slots__ = ("op", "text", "dst", "src", "srcc", "cls", "ws", "line", "asm")

    def __init__(self, op, args, line, asm):
        self.op, self.line, self.asm = op, line, asm
        self.text = f"{op} {args}".strip()
        ops = [a.strip() for a in _split_args(args)]
        self.dst, self.src, self.srcc = set(), set(), set()
        self.ws = 1
        if op == "s_nop":
            self.ws = int(ops[0], 0) + 1 if ops else 1
        if op.startswith("v_mfma"):
            self.cls = "mfma"
            self.dst = _regs(ops[0])
            self.src = _regs(" ".join(ops[1:3]))
            self.srcc = _regs(ops[3]) if len(ops) > 3 else set()
        elif op.startswith("v_"):
            self.cls = "valu"
            if ops and _regs(ops[0]) and not op.startswith(("v_cmp", "v_cmpx")):
                self.dst = _regs(ops[0])
                self.src = _regs(" ".join(ops[1:]))
                if op.startswith(_WRITES_BOTH) and len(ops) > 1:
                    self.dst |= _regs(ops[1])
            else:
                self.src = _regs(" ".join(ops))
        elif op.startswith(("ds_", "global_", "buffer_", "flat_", "scratch_")):
            self.cls = "mem"
            loads = ("read" in op or "load" in op or "_rtn" in op) and "_lds" not in op
            if loads and ops:
                self.dst = _regs(ops[0])
                self.src = _regs(" ".join(ops[1:]))
            else:
                self.src = _regs(" ".join(ops))
        else:
            self.cls = "other"


def _split_args(args):
    out, depth, cur = [], 0, ""
    for ch in args:
        if ch == "[":
            depth += 1
        elif ch == "]":
            depth -= 1
        if ch == "," and depth == 0:
            out.append(cur)
            cur = ""
        else:
            cur += ch
    if cur.strip():
        out.append(cur)
    return out


def _functions(text):
    """(name, [items]) per function; an item is an Ins or ('label', name)."""
    funcs, cur, name, in_asm = [], None, None, False
    for n, raw in enumerate(text.splitlines(), 1):
        line = raw.strip()
        if line.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if line.startswith(";;#ASMEND"):
            in_asm = False
            continue
        code = line.split(";")[0].strip()
        if not code:
            continue
        m = _LABEL.match(code)
        if m:
            lab = m.group(1)
            if not lab.startswith(".") and not lab.startswith("$"):
                name, cur = lab, []
                funcs.append((name, cur))
            elif cur is not None:
                cur.append(("label", lab))
            continue
        if cur is None or code.startswith("."):
            if code.startswith(".end_amdhsa_kernel") or code.startswith(".Lfunc_end"):
                cur = None
            continue
        parts = code.split(None, 1)
        cur.append(Ins(parts[0], parts[1] if len(parts) > 1 else "", n, in_asm))
    return funcs


def _rule(e, l):
    """Wait states needed between earlier e and later l (0 if none)."""
    need = 0
    if e.cls == "valu" and l.cls == "mfma":
        if e.dst & (l.src | l.srcc):
            need = max(need, 2)
    if e.cls == "mfma":
        p = _passes(e.op)
        if l.cls in ("valu", "mem") and e.dst & (l.src | l.dst):
            need = max(need, p + 3)
        if l.cls == "mfma":
            if e.dst & l.src:
                need = max(need, p + 3)
            if e.dst & l.srcc and not (l.srcc == e.dst and l.op == e.op):
                need = max(need, p + 3)
        if l.cls == "valu" and e.srcc & l.dst:
            need = max(need, p - 1)
    return need


def check(text, window=20):
    """Violations as strings: 'function: line a (earlier) .. line b: needs N, has M'."""
    out = []
    for fname, items in _functions(text):
        # basic-block graph: predecessors of every item index
        label_at = {}
        for i, it in enumerate(items):
            if isinstance(it, tuple):
                label_at[it[1]] = i
        preds = {i: [] for i in range(len(items))}
        for i, it in enumerate(items):
            if isinstance(it, tuple):
                continue
            m = _BRANCH.match(it.text)
            if m and m.group(1) in label_at:
                preds[label_at[m.group(1)]].append(i)
        for i, it in enumerate(items):
            if isinstance(it, tuple) or it.cls not in ("valu", "mfma", "mem"):
                continue
            # walk back over every path into it; `jumped` marks a branch
            # reached from its target (an unconditional branch or the end
            # of the program is no fall-through predecessor)
            seen = set()
            stack = [(i - 1, 0, False)]
            while stack:
                j, ws, jumped = stack.pop()
                if j < 0 or ws >= window or (j, ws, jumped) in seen:
                    continue
                seen.add((j, ws, jumped))
                e = items[j]
                if isinstance(e, tuple):
                    stack.append((j - 1, ws, False))
                    for pj in preds[j]:
                        stack.append((pj, ws, True))
                    continue
                if not jumped and e.op in ("s_endpgm", "s_branch", "s_setpc_b64"):
                    continue
                need = _rule(e, it)
                if need > ws and (e.asm or it.asm):
                    out.append(f"{fname}: line {e.line} ({e.text}) .. line {it.line} "
                               f"({it.text}): needs {need} wait states, has {ws}")
                stack.append((j - 1, ws + e.ws, False))
    return out


if __name__ == "__main__":
    bad = check(open(sys.argv[1]).read())
    print("\n".join(bad[:200]))
    print(f"{len(bad)} violation(s)")
