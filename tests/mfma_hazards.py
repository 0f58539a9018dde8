"""Wait-state scan of AMDGPU assembly around MFMA instructions.

The FP4 kernel issues its MFMAs as inline assembly (so that they accumulate
in place), which the compiler does not recognise as MFMAs: it inserts none of
the wait states the matrix-core dependency rules ask for. This scan checks the
built code for them: no instruction may write an MFMA source register within
2 wait states before the MFMA, and no instruction other than a later MFMA
accumulating into the same registers may touch an MFMA's destination within
`after` wait states (the rules ask for at most 18 for the longest MFMAs; the
4-pass FP4 form needs fewer). `s_nop k` counts k + 1 wait states, any other
instruction one. The scan follows the text in order (fall-through), which is
where the compiler places the code between a loop's last MFMA and what reads
its results.
"""
import re

_REG = re.compile(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b")
_NO_DEST = ("ds_write", "global_store", "scratch_store", "buffer_store", "s_", "v_mfma")


def _regs(text):
    out = set()
    for m in _REG.finditer(text):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def _instructions(asm_text):
    out = []
    for line in asm_text.splitlines():
        line = line.split(";")[0].split("//")[0].strip()
        if not line or line.startswith(".") or line.endswith(":"):
            continue
        parts = line.split(None, 1)
        fields = [f.strip() for f in re.split(r",(?![^\[]*\])", parts[1])] if len(parts) > 1 else []
        out.append((parts[0], fields))
    return out


def scan(asm_text, before=2, after=10):
    """List of hazard descriptions (empty: none found) and the MFMA count."""
    ins = _instructions(asm_text)
    found, count = [], 0
    for idx, (op, f) in enumerate(ins):
        if not op.startswith("v_mfma"):
            continue
        count += 1
        dst = _regs(f[0])
        srcs = set().union(*(_regs(x) for x in f[1:])) if len(f) > 1 else set()
        ws, j = 0, idx - 1
        while j >= 0 and ws < before:
            o, g = ins[j]
            if o == "s_nop":
                ws += int(g[0]) + 1
            else:
                if g and not o.startswith(_NO_DEST) and _regs(g[0]) & srcs:
                    found.append(f"{o} {g[0]} writes a source of {op} {f[0]} {ws} wait states before it")
                ws += 1
            j -= 1
        ws, j = 0, idx + 1
        while j < len(ins) and ws < after:
            o, g = ins[j]
            if o == "s_nop":
                ws += int(g[0]) + 1
            else:
                if o.startswith("v_mfma"):
                    if set().union(*(_regs(x) for x in g[1:3])) & dst or (_regs(g[0]) & dst and
                                                                          _regs(g[3]) != _regs(g[0])):
                        found.append(f"{o} reads the result of {op} {f[0]} {ws} wait states after it")
                elif set().union(*(_regs(x) for x in g)) & dst if g else False:
                    found.append(f"{o} {','.join(g)} touches the result of {op} {f[0]} "
                                 f"{ws} wait states after it")
                ws += 1
            j += 1
    return found, count
