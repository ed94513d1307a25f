"""Static check of gfx950 assembly: every MFMA result must be at least NEED
issue slots (instructions, s_nop n counting n + 1) old before a vector ALU
instruction reads it, along every control-flow path, across blocks included.

On gfx950 a v_mfma_f32_16x16x32 result becomes readable 7 slots after the
MFMA issues (measured with register-only probes: a read after 0..6 s_nop
slots returns the register's previous contents).  The compiler pads in-block
reads itself, but once left a result read one slot after a branch whose
skipped block it had counted as padding; this check catches that class."""
from __future__ import annotations

import re
from typing import Dict, List


def _regs(tok: str) -> set:
    tok = tok.strip().rstrip(",")
    m = re.fullmatch(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.fullmatch(r"v(\d+)", tok)
    return {int(m.group(1))} if m else set()


def _parse(ins: str):
    op = ins.split()[0]
    rest = ins[len(op):].split(";")[0]
    toks = [t for t in re.split(r",\s*|\s+", rest.strip()) if t]
    slots = int(toks[0], 0) + 1 if op == "s_nop" and toks else 1
    return op, toks, slots


def functions(asm: str) -> List[Dict]:
    """Functions of an assembly listing split into basic blocks: a block
    ends at a label or after a branch."""
    funcs, cur, blk = [], None, None
    for ln in asm.split("\n"):
        if re.match(r"^_Z\w+:", ln):
            cur = {"name": ln.split(":")[0], "blocks": [], "labels": {}}
            blk = {"label": "entry", "ins": []}
            cur["blocks"].append(blk)
            funcs.append(cur)
            continue
        if cur is None:
            continue
        if ln.startswith(".Lfunc_end"):
            cur = None
            continue
        m = re.match(r"^(\.LBB\w+):", ln)
        if m:
            blk = {"label": m.group(1), "ins": []}
            cur["labels"][m.group(1)] = len(cur["blocks"])
            cur["blocks"].append(blk)
            continue
        s = ln.strip()
        if not s or s.startswith(";") or s.startswith(".") or s.endswith(":"):
            continue
        blk["ins"].append(s)
        op = s.split()[0]
        if op.startswith("s_cbranch") or op == "s_branch":
            blk = {"label": f"after_branch_{len(cur['blocks'])}", "ins": []}
            cur["blocks"].append(blk)
    return funcs


def early_reads(asm: str, need: int = 8, max_depth: int = 6) -> List[str]:
    """Reads of an MFMA result fewer than `need` slots after the MFMA."""
    found = []
    for f in functions(asm):
        B = f["blocks"]
        succ = []
        for i, b in enumerate(B):
            s = []
            last = b["ins"][-1] if b["ins"] else ""
            op = last.split()[0] if last else ""
            if op.startswith("s_cbranch") or op == "s_branch":
                tgt = last.split()[1]
                if tgt in f["labels"]:
                    s.append(f["labels"][tgt])
            if op not in ("s_branch", "s_endpgm", "s_setpc_b64") and i + 1 < len(B):
                s.append(i + 1)
            succ.append(s)
        for bi, b in enumerate(B):
            for ii, ins in enumerate(b["ins"]):
                op, toks, _ = _parse(ins)
                if not op.startswith("v_mfma"):
                    continue
                dst = _regs(toks[0])
                stack, seen = [(bi, ii + 1, 0, 0)], set()
                while stack:
                    cb, ci, w, depth = stack.pop()
                    if (cb, ci, w) in seen or depth > max_depth:
                        continue
                    seen.add((cb, ci, w))
                    seq, stop = B[cb]["ins"], False
                    while ci < len(seq):
                        if w >= need:
                            stop = True
                            break
                        op2, toks2, slots = _parse(seq[ci])
                        if op2.startswith("v_") and not op2.startswith("v_mfma"):
                            src = toks2 if op2.startswith(("v_permlane", "v_accvgpr")) else toks2[1:]
                            read = set().union(*[_regs(t) for t in src]) if src else set()
                            if read & dst:
                                found.append(f"{f['name']}: {ins.split(';')[0].strip()} -> {seq[ci]} "
                                             f"after {w} slots ({B[bi]['label']} -> {B[cb]['label']})")
                                stop = True
                                break
                        w += slots
                        ci += 1
                    if not stop and w < need:
                        for s in succ[cb]:
                            stack.append((s, 0, w, depth + 1))
    return found
