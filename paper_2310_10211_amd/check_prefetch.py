"""Build-time check of the register discipline of the fused training kernel.

The kernel issues its fp32 master prefetches as explicit load instructions
(inline assembly) and waits for them with one explicit ``s_waitcnt vmcnt``
placed where the loaded values are first needed.  The compiler does not track
such loads, so the generated code is only correct if no instruction reads or
writes a destination register of a prefetch on any path between the load and
the next explicit wait.  This module verifies that property on the kernel's
gfx950 assembly, following the control-flow graph (branches and fall-through),
and raises if any path violates it.
"""
from __future__ import annotations

import re

_REG = re.compile(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b")


def _regs(text: str) -> set:
    out = set()
    for m in _REG.finditer(text):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def _is_wait(lines, k) -> bool:
    return lines[k].strip() == ";;#ASMSTART" and k + 1 < len(lines) and "s_waitcnt vmcnt" in lines[k + 1]


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
            seen, stack = set(), [j + 1]
            while stack:
                k = stack.pop()
                if k in seen or k >= len(lines):
                    continue
                seen.add(k)
                if _is_wait(lines, k):
                    continue                       # this path reaches the explicit wait
                t = lines[k].strip()
                if t and not t.startswith(";") and not t.startswith("."):
                    if _regs(t) & dst:
                        bad.append((i, k, t))
                        continue
                stack.extend(successors(k))
            i = j
        i += 1
    return blocks, bad


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
        found[name] = blocks
    if not found:
        raise RuntimeError("no instantiation of the fused kernel in the assembly")
    return found
