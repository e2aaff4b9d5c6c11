"""Build-time check of the compiled MFMA kernels (the library's own gfx950 assembly).

The GEMM and attention kernels read LDS fragments with inline-asm blocks that
must end with ``s_waitcnt lgkmcnt(0)``.  This check scans the assembly of
every kernel whose name starts with the given prefix and fails if any
register written by an asm LDS read is touched before an
``s_waitcnt lgkmcnt(0)`` has retired it -- i.e. if an asm block lost its wait
or the compiler used a result early.
"""
from __future__ import annotations

import re

_ASM_READS = ("ds_read_b128", "ds_read_b64_tr_b16")


def _regs(tok: str):
    m = re.match(r"^([va])\[(\d+):(\d+)\]$", tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"^([va])(\d+)$", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def check_text(asm: str, kernel_prefix: str = "_ZN4lmoe"):
    """Return {kernel: [offending instructions]} for kernels with hazards."""
    lines = asm.split("\n")
    starts = [i for i, l in enumerate(lines) if re.match(rf"^{kernel_prefix}\w*:", l)]
    bad = {}
    for n, s in enumerate(starts):
        e = starts[n + 1] if n + 1 < len(starts) else len(lines)
        name = lines[s].split(":")[0]
        pending, in_asm, hits = set(), False, []
        for l in lines[s + 1:e]:
            t = l.strip()
            if t.startswith(";;#ASMSTART"):
                in_asm = True
                continue
            if t.startswith(";;#ASMEND"):
                in_asm = False
                continue
            if not t or t.startswith(";") or t.startswith("."):
                continue
            op = t.split()[0]
            if op == "s_waitcnt" and "lgkmcnt(0)" in t:
                pending.clear()
                continue
            toks = [x.strip().split()[0] for x in t[len(op):].split(",") if x.strip()]
            touched = set().union(*[_regs(x) for x in toks]) if toks else set()
            if pending & touched:
                hits.append(t)
            if in_asm and op in _ASM_READS and toks:
                pending |= _regs(toks[0])
        if hits:
            bad[name] = hits
    return bad
