"""Build-time check of the register discipline of the streaming kernels (the
fused two-layer training kernel and the hidden-layer kernel).

The kernels issue their fp32 master prefetches as explicit load instructions
(inline assembly) and waits for them with explicit ``s_waitcnt vmcnt(N)``
instructions placed where the loaded values are first needed.  The compiler
does not track such loads, so the generated code is only correct if, on every
path from a prefetch, no instruction reads or writes one of its destination
registers before a wait that covers the prefetch.  Vector memory operations
complete in issue order, so ``s_waitcnt vmcnt(N)`` covers a load once at least
N further vector memory operations have been issued after it on that path.
This module verifies the property on the kernels' gfx950 assembly, following
the control-flow graph (branches and fall-through) and counting the vector
memory operations along each path, and raises if any path violates it.

A second check covers a hazard the compiler's hazard recognizer does not look
for inside inline assembly: on gfx9 a vector memory instruction that reads an
SGPR (the scalar base of a global load or store) needs five wait states after
a VALU instruction (``v_readfirstlane_b32``, ``v_cmp_*``, a carry-out, ...)
wrote that SGPR.  With fewer, the memory instruction may read the register's
previous content as its base address.  ``sgpr_hazards`` follows every path
from each VALU write of an SGPR for five wait states and reports an
inline-assembly memory instruction that reads the register in that window.
"""
from __future__ import annotations

import re

_REG = re.compile(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b")
_VMEM = re.compile(r"^(global|buffer|scratch|flat)_(load|store|atomic)")
_WAIT = re.compile(r"s_waitcnt\b.*\bvmcnt\((\d+)\)")
_CAP = 64


def _regs(text: str) -> set:
    out = set()
    for m in _REG.finditer(text):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def _instruction(line: str) -> str:
    t = line.strip()
    return "" if (not t or t.startswith(";") or t.startswith(".")) else t


def check_function(lines: list) -> tuple:
    """(prefetch blocks, violations) of one function's assembly lines."""
    label_at = {}
    for i, line in enumerate(lines):
        m = re.match(r"^(\.LBB\w+):", line)
        if m:
            label_at[m.group(1)] = i

    def successors(i):
        t = lines[i].strip()
        m = re.match(r"s_cbranch_\w+\s+(\.LBB\w+)", t)
        if m:
            return [label_at[m.group(1)], i + 1]
        m = re.match(r"s_branch\s+(\.LBB\w+)", t)
        if m:
            return [label_at[m.group(1)]]
        if t.startswith("s_endpgm"):
            return []
        return [i + 1]

    blocks, bad = 0, []
    i = 0
    while i < len(lines):
        if lines[i].strip() == ";;#ASMSTART" and "global_load" in lines[i + 1]:
            dst, j = set(), i + 1
            while lines[j].strip() != ";;#ASMEND":
                m = re.match(r"\s*global_load_\w+\s+(v\[\d+:\d+\]|v\d+)", lines[j])
                if m:
                    dst |= _regs(m.group(1))
                j += 1
            blocks += 1
            # state: (line, vector memory operations issued after the prefetch, capped)
            seen, stack = set(), [(j + 1, 0)]
            while stack:
                k, younger = stack.pop()
                if (k, younger) in seen or k >= len(lines):
                    continue
                seen.add((k, younger))
                t = _instruction(lines[k])
                if t:
                    w = _WAIT.search(t)
                    if w and younger >= int(w.group(1)):
                        continue                   # this path waits for the prefetch here
                    if _VMEM.match(t):
                        younger = min(younger + 1, _CAP)
                    if _regs(t) & dst and not w:
                        bad.append((i, k, t))
                        continue
                stack.extend((n, younger) for n in successors(k))
            i = j
        i += 1
    return blocks, bad


_SREG = re.compile(r"\bs\[(\d+):(\d+)\]|\bs(\d+)\b")
# VALU instructions whose second operand is an SGPR destination (a carry-out or a scale flag)
_SDST2 = re.compile(r"^v_(add_co|sub_co|subrev_co|addc_co|subb_co|subbrev_co)_u32|^v_div_scale|^v_mad_[ui]64")
_VALU_SGPR_WAIT_STATES = 5


def _sregs(text: str) -> set:
    out = set()
    for m in _SREG.finditer(text):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def _operands(t: str) -> list:
    parts = t.split(None, 1)
    return [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []


def _valu_sgpr_writes(t: str) -> set:
    """SGPRs a VALU instruction writes (empty for other instructions)."""
    if not t.startswith("v_"):
        return set()
    ops = _operands(t)
    mnem = t.split(None, 1)[0]
    out = set()
    if ops and _SREG.fullmatch(ops[0]):
        out |= _sregs(ops[0])
    if len(ops) > 1 and _SDST2.match(mnem) and _SREG.fullmatch(ops[1]):
        out |= _sregs(ops[1])
    return out


def sgpr_hazards(lines: list) -> list:
    """(writer line, reader line, reader) of every inline-assembly vector memory
    instruction that reads an SGPR fewer than five wait states after a VALU
    instruction wrote it, on some path."""
    label_at, in_asm = {}, []
    inside = False
    for i, line in enumerate(lines):
        m = re.match(r"^(\.LBB\w+):", line)
        if m:
            label_at[m.group(1)] = i
        t = line.strip()
        if t == ";;#ASMSTART":
            inside = True
        elif t == ";;#ASMEND":
            inside = False
        in_asm.append(inside)

    def successors(i):
        t = lines[i].strip()
        m = re.match(r"s_cbranch_\w+\s+(\.LBB\w+)", t)
        if m:
            return [label_at[m.group(1)], i + 1]
        m = re.match(r"s_branch\s+(\.LBB\w+)", t)
        if m:
            return [label_at[m.group(1)]]
        if t.startswith("s_endpgm"):
            return []
        return [i + 1]

    bad = []
    for i, line in enumerate(lines):
        t = _instruction(line)
        regs = _valu_sgpr_writes(t) if t else set()
        if not regs:
            continue
        seen, stack = set(), [(n, 0) for n in successors(i)]
        while stack:
            k, ws = stack.pop()
            if (k, ws) in seen or k >= len(lines) or ws >= _VALU_SGPR_WAIT_STATES:
                continue
            seen.add((k, ws))
            u = _instruction(lines[k])
            if not u:
                stack.extend((n, ws) for n in successors(k))
                continue
            if in_asm[k] and _VMEM.match(u) and _sregs(" ".join(_operands(u)[1:])) & regs:
                bad.append((i, k, u))
                continue
            m = re.match(r"s_nop\s+(\d+)", u)
            step = int(m.group(1)) + 1 if m else 1
            stack.extend((n, ws + step) for n in successors(k))
    return bad


def check_assembly(asm: str, kernel_prefix: str = "_ZN4gevo8k_fused2") -> dict:
    """Check every instantiation of the kernel; returns {symbol: prefetch blocks}."""
    found = {}
    for m in re.finditer(r"^(" + re.escape(kernel_prefix) + r"\w*):", asm, re.M):
        name = m.group(1)
        end = asm.index(".Lfunc_end", m.end())
        blocks, bad = check_function(asm[m.end():end].split("\n"))
        if bad:
            i, k, t = bad[0]
            raise RuntimeError(f"{name}: a prefetch register is used before its wait "
                               f"({len(bad)} uses; first: {t!r})")
        if blocks == 0:
            raise RuntimeError(f"{name}: no prefetch blocks found; the check no longer matches the kernel")
        haz = sgpr_hazards(asm[m.end():end].split("\n"))
        if haz:
            raise RuntimeError(f"{name}: an inline-assembly memory instruction reads an SGPR fewer than "
                               f"{_VALU_SGPR_WAIT_STATES} wait states after a VALU instruction wrote it "
                               f"({len(haz)} sites; first: {haz[0][2]!r})")
        found[name] = blocks
    if not found:
        raise RuntimeError(f"no instantiation of {kernel_prefix} in the assembly")
    return found


def check_scalar_operands(asm: str, kernel_prefix: str) -> dict:
    """Kernels whose inline-assembly loads take scalar operands (a scalar base
    address, and m0 as the LDS address of a direct-to-LDS load): every such
    operand must be an SGPR (a vector register in ``s_mov_b32 m0, ...`` would
    not be a scalar value; ``vcc_lo`` is an SGPR), and the SGPR hazard check
    must pass.  Returns
    {symbol: number of direct-to-LDS loads}."""
    found = {}
    for m in re.finditer(r"^(" + re.escape(kernel_prefix) + r"\w*):", asm, re.M):
        name = m.group(1)
        end = asm.index(".Lfunc_end", m.end())
        lines = asm[m.end():end].split("\n")
        bad = [t for t in (l.strip() for l in lines) if re.match(r"s_mov_b32\s+m0,\s*v(\d|\[)", t)]
        if bad:
            raise RuntimeError(f"{name}: m0 is written from a vector register ({bad[0]!r})")
        haz = sgpr_hazards(lines)
        if haz:
            raise RuntimeError(f"{name}: an inline-assembly memory instruction reads an SGPR fewer than "
                               f"{_VALU_SGPR_WAIT_STATES} wait states after a VALU instruction wrote it "
                               f"({len(haz)} sites; first: {haz[0][2]!r})")
        found[name] = sum(1 for l in lines if "global_load_lds_" in l)
    if not found:
        raise RuntimeError(f"no instantiation of {kernel_prefix} in the assembly")
    return found
