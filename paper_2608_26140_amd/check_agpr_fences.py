"""Build-time check of the 4-wave GEMM's inline-asm MFMAs (AMD assembly of
this library's own kernels).  The compiler's hazard recognizer does not look
inside inline asm, so the wait states it would insert after an MFMA are the
kernel's own business.  On every path through the kernel's basic blocks
this counts wait states (one per instruction, k + 1 for s_nop k) and flags

  * an instruction other than an MFMA that names an accumulator register
    (a read, a write, a spill) fewer than 19 wait states after an MFMA
    (the most any gfx950 MFMA needs before its result registers are
    touched by other instructions);
  * an MFMA fewer than 4 wait states after another instruction wrote an
    accumulator register (VALU write before MFMA operand read needs 2).

    python -m paper_2608_26140_amd.check_agpr_fences [ASM_FILE]

Without an argument it compiles k_gemm.hip to assembly (hipcc -S) first.
Exits non-zero and lists the offending lines if it finds any."""

from __future__ import annotations

import os
import re
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))


def kernels(asm: str):
    """(name, lines) of every gemm_bf16_w4_kernel instantiation."""
    out, cur, name = [], None, None
    for line in asm.splitlines():
        m = re.match(r"^(_Z\S*gemm_bf16_w4_kernel\S*):", line)
        if m:
            cur, name = [], m.group(1)
            continue
        if cur is not None:
            cur.append(line)
            if "s_endpgm" in line:
                out.append((name, cur))
                cur = None
    return out


MFMA_WAIT = 19   # wait states from an MFMA to other users of its registers
WRITE_WAIT = 4   # wait states from an accumulator write to an MFMA
FAR = 1 << 20

AREG = re.compile(r"\ba(\d+|\[\d+:\d+\])")


def blocks_of(lines):
    """Basic blocks as lists of (line index, instruction), the label map,
    and each block's successors."""
    blocks, labels, cur = [], {}, []
    for i, l in enumerate(lines):
        t = l.split(";")[0].strip()
        m = re.match(r"^(\.LBB\w+):", t)
        if m:
            if cur:
                blocks.append(cur)
            labels[m.group(1)] = len(blocks) if not cur else len(blocks)
            cur = []
            continue
        if not t or t.startswith("."):
            continue
        cur.append((i, t))
        if t.startswith(("s_branch", "s_cbranch", "s_endpgm", "s_setpc")):
            blocks.append(cur)
            cur = []
    if cur:
        blocks.append(cur)
    succ = []
    for k, b in enumerate(blocks):
        last = b[-1][1] if b else ""
        out = []
        m = re.match(r"s_c?branch\w*\s+(\.LBB\w+)", last)
        if m and m.group(1) in labels:
            out.append(labels[m.group(1)])
        if not last.startswith(("s_branch", "s_endpgm", "s_setpc")) and k + 1 < len(blocks):
            out.append(k + 1)
        succ.append(out)
    return blocks, succ


def waits(t):
    m = re.match(r"s_nop\s+(\d+)", t)
    return int(m.group(1)) + 1 if m else 1


def unfenced(lines):
    """(line index, instruction, reason) of every hazard on some path."""
    blocks, succ = blocks_of(lines)

    def scan(k, state, report=None):
        since_mfma, since_write = state
        for i, t in blocks[k]:
            if t.startswith("v_mfma"):
                if since_write < WRITE_WAIT and report is not None:
                    report.append((i, t, f"MFMA {since_write} wait states after an accumulator write"))
                since_mfma, since_write = 0, since_write + 1
                continue
            names_acc = bool(AREG.search(t.split(None, 1)[1] if " " in t else ""))
            if names_acc and since_mfma < MFMA_WAIT and report is not None:
                report.append((i, t, f"{since_mfma} wait states after an MFMA"))
            w = waits(t)
            since_mfma = min(FAR, since_mfma + w)
            since_write = min(FAR, since_write + w)
            if names_acc:
                dst = t.split(None, 1)[1].split(",")[0] if " " in t else ""
                if AREG.search(dst) and not t.startswith(("scratch_store", "buffer_store", "global_store", "ds_write")):
                    since_write = 0
        return since_mfma, since_write

    entry = [(FAR, FAR)] * len(blocks)
    entry[0] = (FAR, FAR)
    reached = [False] * len(blocks)
    reached[0] = True
    work = [0]
    while work:
        k = work.pop()
        out = scan(k, entry[k])
        for n in succ[k]:
            new = (min(entry[n][0], out[0]), min(entry[n][1], out[1]))
            if not reached[n] or new != entry[n]:
                reached[n] = True
                entry[n] = new
                work.append(n)
    bad = []
    for k in range(len(blocks)):
        if reached[k]:
            scan(k, entry[k], bad)
    return bad


def main(argv):
    if argv:
        asm = open(argv[0]).read()
    else:
        from paper_2608_26140_amd.build import FLAGS, HIPCC
        with tempfile.TemporaryDirectory() as d:
            out = os.path.join(d, "k_gemm.s")
            subprocess.run([HIPCC, *FLAGS, "--cuda-device-only", "-S", "-o", out, os.path.join(PKG, "csrc", "k_gemm.hip")],
                           check=True, stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
            asm = open(out).read()
    ks = kernels(asm)
    failed = False
    for name, lines in ks:
        bad = unfenced(lines)
        if bad:
            failed = True
            print(f"{name}: {len(bad)} hazards, e.g.")
            for i, t, why in bad[:5]:
                print(f"  line {i}: {t}  ({why})")
    print(f"checked {len(ks)} kernels: {'FAIL' if failed else 'ok'}")
    return 1 if failed else 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
