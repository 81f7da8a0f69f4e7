"""Static checks of the gfx950 assembly the compiler writes for this
library's kernels (test infrastructure; reads only code built here).

mfma_result_reads(path) walks every control-flow path from each v_mfma to
the first non-MFMA instruction that reads one of its destination registers,
and reports the fewest wait states (instructions issued in between, an
`s_nop N` counting N + 1) on any path, with the reading instruction."""
import collections
import re

_STORE_PREFIXES = ("global_store", "buffer_store", "flat_store", "scratch_store", "ds_write", "ds_store")


def regs(tok):
    m = re.match(r"([va])\[(\d+):(\d+)\]$", tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"([va])(\d+)$", tok)
    if m:
        return {(m.group(1), int(m.group(2)))}
    return set()


def _split(s):
    parts = s.split(None, 1)
    ops = [o.strip() for o in re.split(r",\s*", parts[1])] if len(parts) > 1 else []
    return parts[0], ops


def _sources(op, ops):
    if op.startswith(_STORE_PREFIXES) or op.startswith("s_"):
        return set().union(*[regs(o) for o in ops]) if ops else set()
    return set().union(*[regs(o) for o in ops[1:]]) if len(ops) > 1 else set()


def _dest(op, ops):
    if op.startswith(_STORE_PREFIXES) or op.startswith("s_") or not ops:
        return set()
    return regs(ops[0])


def functions(path):
    """{kernel symbol: [instruction lines]} of an assembly file."""
    out, fn = {}, None
    with open(path) as fh:
        for line in fh:
            s = line.split(";")[0].strip()
            m = re.match(r"^(_Z\w+):$", s)
            if m:
                fn = m.group(1)
                out[fn] = []
                continue
            if fn is None or not s:
                continue
            if s.startswith(".Lfunc_end"):
                fn = None
                continue
            if s.startswith(".") and not s.endswith(":"):
                continue
            out[fn].append(s)
    return out


def _cfg(lines):
    blocks, order, cur = collections.OrderedDict(), [], "__entry"
    blocks[cur] = []
    order.append(cur)
    anon = 0
    for s in lines:
        if s.endswith(":"):
            cur = s[:-1]
            blocks[cur] = []
            order.append(cur)
        else:
            op, ops = _split(s)
            blocks[cur].append((op, ops))
            if op.startswith(("s_cbranch", "s_branch")):
                # a branch ends its basic block; the fall-through starts a new one
                anon += 1
                cur = "__fall%d" % anon
                blocks[cur] = []
                order.append(cur)
    succ = {}
    for i, b in enumerate(order):
        nxt, s, ends = (order[i + 1] if i + 1 < len(order) else None), [], False
        for op, ops in blocks[b]:
            if op.startswith("s_cbranch"):
                s.append(ops[0])
            elif op == "s_branch":
                s.append(ops[0])
                ends = True
            elif op == "s_endpgm":
                ends = True
        if not ends and nxt:
            s.append(nxt)
        succ[b] = [x for x in s if x in blocks]
    return order, blocks, succ


def mfma_result_reads(lines, cap=64):
    """[(wait states, mfma, reading instruction or None)] for every v_mfma of
    one kernel (None: no read within `cap` wait states on any path)."""
    order, blocks, succ = _cfg(lines)
    out = []
    for b in order:
        for idx, (op, ops) in enumerate(blocks[b]):
            if not op.startswith("v_mfma"):
                continue
            dst = regs(ops[0])
            best = [cap, None]
            stack, seen = [(b, idx + 1, 0, frozenset(dst))], {}
            while stack:
                bb, ii, ws, live = stack.pop()
                if ws >= best[0] or (seen.get((bb, ii, live), 1 << 30) <= ws):
                    continue
                seen[(bb, ii, live)] = ws
                ins, stop = blocks[bb], False
                while ii < len(ins):
                    op2, ops2 = ins[ii]
                    if op2 == "s_endpgm":
                        stop = True
                        break
                    if op2.startswith("v_mfma"):
                        # A dependent MFMA (srcC) is interlocked by the hardware.
                        live = live - (_dest(op2, ops2) - _sources(op2, ops2))
                        ws += 1
                    else:
                        if _sources(op2, ops2) & live:
                            if ws < best[0]:
                                best[:] = [ws, op2]
                            stop = True
                            break
                        live = live - _dest(op2, ops2)
                        ws += int(ops2[0], 0) + 1 if op2 == "s_nop" else 1
                    if not live or ws >= best[0]:
                        stop = True
                        break
                    ii += 1
                if not stop:
                    stack.extend((s, 0, ws, live) for s in succ[bb])
            out.append((best[0], op, best[1], "agpr" if any(r[0] == "a" for r in dst) else "vgpr"))
    return out
