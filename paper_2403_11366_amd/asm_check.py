"""Build-time check of the kernels that issue LDS reads as inline assembly.

Some GEMM pipelines issue their LDS fragment reads as inline assembly and wait
for them with hand-counted `s_waitcnt lgkmcnt(N)` (the compiler would
otherwise wait for every global-to-LDS copy in flight before each read).  The
compiler treats the asm's destination registers as written the moment the
asm statement ends, so the result is correct only if nothing touches those
registers before the wait that covers the read: no copy, no spill to scratch,
no call that passes them through memory.  This module reads the gfx950
assembly the build saved (`-save-temps=obj`) and checks, for every function
that contains inline-asm LDS reads:

  * no scratch access and no call anywhere in the function;
  * along the instruction stream, no instruction other than an `s_waitcnt`
    reads or writes a register that is the destination of an LDS read still
    outstanding (LDS operations complete in issue order, so `lgkmcnt(N)`
    retires all but the newest N);
  * no LDS read is outstanding at a branch or a label (the check follows
    straight-line code only, so the pipelines must drain at stage ends).

Usage: python -m paper_2403_11366_amd.asm_check FILE.s [...]; build() calls
check_files() on the saved assembly and fails the build on any finding.
"""
from __future__ import annotations

import re
import subprocess
import sys

_FUNC = re.compile(r"^(_Z\S+):")
_REG = re.compile(r"\b([vas])(?:\[(\d+):(\d+)\]|(\d+)\b)")
_LGKM = re.compile(r"lgkmcnt\((\d+)\)")


def _regs(operands: str):
    out = set()
    for kind, lo, hi, one in _REG.findall(operands):
        if kind == "s":
            continue
        if one:
            out.add((kind, int(one)))
        else:
            out.update((kind, i) for i in range(int(lo), int(hi) + 1))
    return out


def _demangle(name: str) -> str:
    try:
        return subprocess.run(["c++filt", name], capture_output=True, text=True).stdout.strip() or name
    except OSError:
        return name


def check_function(name: str, lines: list) -> list:
    """Findings for one function's assembly lines (empty if it has no
    inline-asm LDS reads or passes)."""
    if not has_asm_reads(lines):
        return []
    errs = []
    # outstanding LDS operations in issue order: (line, destination registers,
    # issued by inline asm).  Reads the compiler issued itself are counted (they
    # share the counter) but their waits are the compiler's own business.
    pending = []
    in_asm = False
    for no, ln in enumerate(lines):
        t = ln.strip()
        if t.startswith(";;#ASMSTART"):
            in_asm = True
        elif t.startswith(";;#ASMEND"):
            in_asm = False
        s = ln.split(";")[0].strip()
        if not s or s.startswith("."):
            if re.match(r"^\.LBB\S*:", t) and any(a for _, _, a in pending):
                errs.append(f"{name}: inline-asm LDS reads outstanding at label {t.split()[0]} (line {no})")
            if re.match(r"^\.LBB\S*:", t):
                pending = []
            continue
        op, _, rest = s.partition(" ")
        if op.startswith("scratch_") or op in ("s_swappc_b64", "s_setpc_b64") or "off, off offset" in s:
            errs.append(f"{name}: {op} at line {no}")
        if op == "s_waitcnt":
            m = _LGKM.search(rest)
            if m:
                keep = int(m.group(1))
                while len(pending) > keep:
                    pending.pop(0)
            continue
        if op.startswith("s_cbranch") or op == "s_branch":
            if any(a for _, _, a in pending):
                errs.append(f"{name}: inline-asm LDS reads outstanding at a branch (line {no})")
            continue
        regs = _regs(rest)
        busy = set()
        for _, d, a in pending:
            if a:
                busy |= d
        hit = regs & busy
        if hit:
            errs.append(f"{name}: line {no} `{s}` touches {sorted(hit)[:4]} before its LDS read completed")
        if op.startswith("ds_"):
            dest = set()
            if op.startswith("ds_read") or "rtn" in op:
                dest = _regs(rest.split(",")[0])
            pending.append((no, dest, in_asm))
    return errs


def check_assembly(text: str) -> list:
    lines = text.split("\n")
    errs = []
    name, body = None, []
    for ln in lines:
        m = _FUNC.match(ln)
        if m:
            name, body = m.group(1), []
            continue
        if name and ln.strip().startswith(".Lfunc_end"):
            errs += check_function(_demangle(name), body)
            name = None
            continue
        if name:
            body.append(ln)
    return errs


def check_files(paths) -> list:
    errs = []
    for p in paths:
        with open(p) as f:
            errs += check_assembly(f.read())
    return errs


def has_asm_reads(lines) -> bool:
    """True if an inline-asm block of these assembly lines issues an LDS read."""
    in_asm = False
    for ln in lines:
        s = ln.strip()
        if s.startswith(";;#ASMSTART"):
            in_asm = True
        elif s.startswith(";;#ASMEND"):
            in_asm = False
        elif in_asm and s.startswith("ds_read"):
            return True
    return False


def count_checked_text(text: str) -> int:
    """Number of functions with inline-asm LDS reads in one assembly listing."""
    return sum(1 for chunk in re.split(r"\n(?=_Z\S+:)", text) if has_asm_reads(chunk.split("\n")))


def count_checked(paths) -> int:
    """Number of functions with inline-asm LDS reads in these files."""
    n = 0
    for p in paths:
        with open(p) as f:
            n += count_checked_text(f.read())
    return n


if __name__ == "__main__":
    found = check_files(sys.argv[1:])
    for e in found:
        print(e)
    print(f"{count_checked(sys.argv[1:])} function(s) with inline-asm LDS reads, {len(found)} finding(s)")
    sys.exit(1 if found else 0)
