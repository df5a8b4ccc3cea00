"""Static check of gfx950 assembly for one matrix-core hazard.

A matrix (MFMA/XDL) instruction writes its result several cycles after it
issues; a vector-ALU, memory or LDS instruction that reads the result must
come enough instructions later, and on gfx950 the compiler inserts the
s_nop padding.  We have seen the padding missing on one control-flow path:
a product followed by a conditional branch whose target read the result two
instructions later (the fall-through path was padded), which returned stale
registers on the GPU now and then.  This module walks every path of up to a
few branches from each product and reports reads that come sooner than the
spacing the compiler itself uses inside a basic block (4 + the instruction's
passes: 8 for the 16x16 shapes, 12 for the 32x32 ones).

Used by tests/test_isa_hazards.py on the library sources compiled with -S.
"""
import re

# required instructions between a product and a read of its result
SPACING = {"16x16": 8, "32x32": 12, "4x4": 6}

_LABEL = re.compile(r"^(\.?[A-Za-z_][\w.$]*):")
_FUNC = re.compile(r"^(_Z\w+):")


def _regs(tok):
    """Registers named by an operand, as (file, index): v (vector) or a
    (accumulation)."""
    m = re.match(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), n) for n in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"([va])(\d+)$", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def _parse(line):
    body = line.split(";")[0].strip()
    if not body or body.startswith(".") or body.endswith(":"):
        return None, []
    parts = body.split(None, 1)
    ops = [o.strip() for o in parts[1].split(",")] if len(parts) > 1 else []
    return parts[0], ops


_STORES = ("global_store", "buffer_store", "ds_write", "flat_store", "scratch_store")


def scan(text, max_depth=4):
    """Findings (function, product line, read line, spacing, read text) in
    the assembly `text`."""
    lines = text.split("\n")
    labels = {}
    for i, l in enumerate(lines):
        m = _LABEL.match(l)
        if m:
            labels[m.group(1)] = i
    findings = []

    def walk(i, dst, need, dist, depth, seen, origin):
        while i < len(lines) and dist < need:
            if _FUNC.match(lines[i]):
                return
            op, ops = _parse(lines[i])
            if op is None:
                i += 1
                continue
            if op == "s_endpgm":
                return
            if op.startswith("v_mfma"):
                if ops and _regs(ops[0]) & dst:      # result overwritten
                    return
                dist += 1
                i += 1
                continue
            srcs = set()
            for o in (ops if op.startswith(_STORES) else ops[1:]):
                srcs |= _regs(o)
            if op.startswith(("v_", "global_", "buffer_", "ds_", "flat_", "scratch_")) and srcs & dst:
                findings.append((origin[0], origin[1] + 1, i + 1, dist, lines[i].strip()))
                return
            if op.startswith("v_") and ops and _regs(ops[0]) >= dst:
                return
            dist += int(ops[0], 0) + 1 if op == "s_nop" else 1
            if op.startswith("s_cbranch") or op == "s_branch":
                tgt = ops[0] if ops else ""
                if tgt in labels and depth < max_depth and (tgt, dist) not in seen:
                    seen.add((tgt, dist))
                    walk(labels[tgt] + 1, dst, need, dist, depth + 1, seen, origin)
                if op == "s_branch":
                    return
            i += 1

    func = None
    for i, l in enumerate(lines):
        m = _FUNC.match(l)
        if m:
            func = m.group(1)
        op, ops = _parse(l)
        if op and op.startswith("v_mfma") and ops:
            need = next((v for k, v in SPACING.items() if k in op), 12)
            walk(i + 1, _regs(ops[0]), need, 0, 0, set(), (func, i))
    # one finding per (product, read), the shortest path
    best = {}
    for f in findings:
        k = (f[0], f[1], f[2])
        if k not in best or f[3] < best[k][3]:
            best[k] = f
    return sorted(best.values(), key=lambda f: (f[1], f[2]))
